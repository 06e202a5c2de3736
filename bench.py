#!/usr/bin/env python
"""Benchmark of the forked-decode hot path on one MI355X.

One step = one pass of the whole hot path over the workload's batch: the
cascade partial attention over every fork group's shared prefix and every
thread's private range (main decode rows, probe decode rows and the main
threads' verify rows with the causal rule over the drafts), the log-sum-exp
merge, the greedy argmax over the verify logits and the longest-prefix
accept. The copy-on-write forks, appends and the plan are host work done once
per fork, before the timed region; their host time is reported beside it.

Default workload: the Qwen3-30B-A3B-shaped mixed batch (32 query / 4 KV heads,
head dim 128, bf16, block size 16; 64 sessions x (main + 2 probes), 32768-token
shared prefixes, log-uniform private suffixes in [1, 4096], mains verify K=8
drafts in the same batch, vocabulary 151936), seeded synthetic data.

Prints one JSON line. ``value`` is unique-KV GB/s: each shared prefix counted
once, each private range once, over the median step time (inputs resident in
HBM). Each timed step is preceded by a 512 MiB scratch write and a 512 MiB
read of another buffer, which evict the caches, and timed alone with HIP
events; the minimum, the mean and the rate of the same steps run back to back
are reported beside the median. ``roofline``
reports the dominant kernel (the partial attention) from HIP events recorded
around its launches in the timed region; ``read_ceiling`` is the best rate of
plain streaming-read kernels measured in the same process.
"""
import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "forked decode-attn unique-KV GB/s (% of 8 TB/s) + verified tokens/s"
HBM_PEAK_GBPS = 8000.0
# Dense MFMA peaks of MI355X (no sparsity), TFLOP/s, by the kernel's operand type.
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
DEFAULT_WORKLOAD = "qwen3-30b-a3b-mixed"
FLUSH_BYTES = 512 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_partial_traffic.json")
# the attention kernel's source and every header it includes
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2607_03333_amd", "csrc", f)
                  for f in ("attention.hip", "device_common.h", "kernels.h", "plan_types.h")]


def kernel_source_hash():
    """First 16 hex digits of the sha256 of the attention kernel's code
    (KERNEL_SOURCES with comments and whitespace removed): counters taken on
    one code stay valid across comment edits and no longer match once the
    code changes."""
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per attention launch from the rocprofv3 counter runs, if they
    were taken on the current kernel source for this workload."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256_16") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t.get("bytes_per_launch")


def attention_flops(wl, index, spec):
    """Algorithmic flops of one step's attention: Q.K^T and P.V cost 2 D
    flops each per (query-head row, visible position). A thread's rows are
    the last positions of its context, each seeing the positions up to its
    own (causal)."""
    total = 0
    for seq, r in zip(spec.seqs, spec.n_rows):
        n = wl.thread_len(seq, index)
        visible = r * (n - r + 1) + r * (r - 1) // 2
        total += visible
    return total * wl.hq * 4 * wl.d


def read_ceiling(torch, spork, nbytes=2 << 30, reps=10):
    """The device's attainable read bandwidth: the plain streaming-read
    kernels over ``nbytes`` (register loads and direct-to-LDS loads in the
    attention kernel's ring shape, each with the default and the
    non-temporal cache policy, at 512 and 1024 workgroups); the best median
    over ``reps`` launches is the ceiling. Also brings the GPU to its
    working clocks before the benchmark's warm-up."""
    import numpy as np
    dev = torch.device("cuda:0")
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    src.fill_(1)
    sink = torch.empty(1024 * 256, dtype=torch.int32, device=dev)
    names = {0: "register loads", 1: "direct-to-LDS ring", 2: "register loads, non-temporal",
             3: "direct-to-LDS ring, non-temporal"}
    results = []
    for mode in (0, 1, 2, 3):
        for grid in (512, 1024):
            for _ in range(3):
                spork.spork_read_ceiling(src, nbytes, grid, mode, sink)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
            for a, b in ev:
                a.record()
                spork.spork_read_ceiling(src, nbytes, grid, mode, sink)
                b.record()
            torch.cuda.synchronize()
            ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
            results.append({"mode": names[mode], "grid": grid, "gbps": round(nbytes / (ms * 1e-3) / 1e9, 1)})
    del src, sink
    best = max(results, key=lambda r: r["gbps"])
    return {"gbps": best["gbps"], "kernel": f"{best['mode']}, {best['grid']} workgroups", "bytes": nbytes,
            "all": results}


def cpu_baseline(wl, step_specs, target_s, single_core=False):
    """The oracle, untuned, on whole sessions of the same workload until about
    ``target_s`` seconds of CPU work (passes over all sessions repeat for a
    workload that takes less); GB/s on the same unique-KV accounting. BLAS
    runs on every core it sees, or on one with ``single_core``."""
    from threadpoolctl import threadpool_info, threadpool_limits

    with threadpool_limits(1 if single_core else None):
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        return _cpu_baseline(wl, step_specs, target_s, threads)


def _cpu_baseline(wl, step_specs, target_s, threads):
    import oracle
    from paper_2607_03333_amd import synth

    per_tok = 2 * wl.hkv * wl.d * (2 if wl.dtype == synth.BF16 else 4)
    sessions = sorted({t.session for t in wl.threads})
    done, nbytes, rows, t0 = 0, 0, 0, time.perf_counter()
    passes = 0
    while True:
        for s in sessions:
            done, nbytes, rows = _oracle_session(wl, step_specs, s, per_tok, done, nbytes, rows, oracle, synth)
            if time.perf_counter() - t0 >= target_s:
                break
        passes += 1
        if time.perf_counter() - t0 >= target_s:
            break
    dt = time.perf_counter() - t0
    what = (f"{done} of {len(sessions)} sessions" if done <= len(sessions)
            else f"{done} session runs, {done / len(sessions):.1f} passes over all {len(sessions)} sessions")
    return {"value": nbytes / dt / 1e9, "unit": "GB/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{what} ({rows} query rows, {nbytes} unique KV bytes) in {dt:.1f} s, float64 NumPy, "
                      f"{os.cpu_count()} logical CPUs visible"}


def _oracle_session(wl, step_specs, s, per_tok, done, nbytes, rows, oracle, synth):
    """The oracle over one session's threads in every step: gather, attention,
    argmax and accept. Returns the updated counts."""
    if True:
        for si, st in step_specs:
            row = 0
            vrow = 0
            for seq, n in zip(st.seqs, st.n_rows):
                th = next(t for t in wl.threads if t.seq == seq)
                if th.session == s:
                    L = wl.thread_len(seq, si)
                    k, v = wl.context(seq, L)
                    oracle.attend(synth.to_f64(st.q[row:row + n], wl.dtype), synth.to_f64(k, wl.dtype),
                                  synth.to_f64(v, wl.dtype), wl.sm_scale)
                    nbytes += (L - wl.prefix_len[s]) * per_tok
                    rows += n
                    if st.verify_k and th.drafts:
                        kk = st.verify_k
                        g = oracle.argmax_rows(synth.to_f64(st.logits[vrow * (kk + 1):(vrow + 1) * (kk + 1)],
                                                            wl.logits_dtype))
                        oracle.accept_drafts(g, st.drafts[vrow:vrow + 1])
                if th.drafts and st.verify_k:
                    vrow += 1
                row += n
            nbytes += wl.prefix_len[s] * per_tok
        return done + 1, nbytes, rows


def confidence_bench(args, torch, spork, synth):
    """D2 confidence gate alone: one JSON line, HBM roofline of the chunk pass
    (2 bytes per bf16 logit read once)."""
    vocab = 151936
    b = synth.probe_batch(args.confidence_probes, vocab, dtype=synth.BF16, span=(0, 16), seed=1)
    rows = b.logits.shape[0]
    dev = torch.device("cuda:0")
    x = torch.from_numpy(b.logits.view("int16")).to(dev).view(torch.bfloat16)
    off = torch.from_numpy(b.span_off).to(dev)
    am = torch.empty(rows, dtype=torch.int32, device=dev)
    lp = torch.empty(rows, dtype=torch.float32, device=dev)
    conf = torch.empty(args.confidence_probes, dtype=torch.float32, device=dev)
    commit = torch.empty(args.confidence_probes, dtype=torch.int32, device=dev)
    ws = torch.empty(spork.spork_confidence_workspace_bytes(rows, vocab), dtype=torch.uint8, device=dev)

    def step():
        spork.spork_probe_confidence(x, spork.SPORK_DTYPE_BF16, vocab, rows, off, args.confidence_probes,
                                     0.90, am, lp, conf, commit, ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    spork.spork_timing_read()
    spork.spork_timing_enable(True)
    start.record(stream)
    for _ in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    spork.spork_timing_enable(False)
    kern = spork.spork_timing_read()
    ms_step = start.elapsed_time(end) / args.steps
    nbytes = rows * vocab * 2
    ms_chunks = kern["conf_chunks"][0] / max(kern["conf_chunks"][1], 1)
    achieved = nbytes / (ms_chunks * 1e-3) / 1e9
    print(json.dumps({
        "metric": "D2 confidence gate: logits GB/s", "value": round(nbytes / (ms_step * 1e-3) / 1e9, 2),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded Gaussian logits with a boosted top-1 token)",
        "config": {"workload": "probe-confidence", "probes": args.confidence_probes, "rows": rows,
                   "vocab": vocab, "theta": 0.90},
        "kernel_ms_per_step": {k: round(v[0] / max(v[1], 1), 4) for k, v in kern.items() if v[1]},
        "commits": int(commit.sum().item()),
        "roofline": {"bound": "hbm", "kernel": "conf_chunks", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                     "avg_launch_ms": round(ms_chunks, 4), "algorithmic_bytes_per_launch": nbytes}}), flush=True)


def ngram_bench(args, torch, spork, synth):
    """n-gram draft proposer alone: one JSON line, HBM roofline of the scan
    (4 bytes per token read once)."""
    import numpy as np
    n = args.ngram_seqs
    tok, off = synth.token_histories(n, (32768, 36864), seed=1)
    dev = torch.device("cuda:0")
    t = torch.from_numpy(tok).to(dev)
    o = torch.from_numpy(off).to(dev)
    k, n_min, n_max = 8, 2, 4
    max_len = int(np.diff(off).max())
    drafts = torch.empty(n * k, dtype=torch.int32, device=dev)
    cnt = torch.empty(n, dtype=torch.int32, device=dev)
    ws = torch.empty(spork.spork_ngram_workspace_bytes(n, max_len), dtype=torch.uint8, device=dev)

    def step():
        spork.spork_ngram_propose(t, o, n, max_len, n_min, n_max, k, drafts, cnt, ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    spork.spork_timing_read()
    spork.spork_timing_enable(True)
    start.record(stream)
    for _ in range(args.steps):
        step()
    end.record(stream)
    torch.cuda.synchronize()
    spork.spork_timing_enable(False)
    kern = spork.spork_timing_read()
    ms_step = start.elapsed_time(end) / args.steps
    nbytes = int(tok.size) * 4
    ms_scan = kern["ngram_scan"][0] / max(kern["ngram_scan"][1], 1)
    achieved = nbytes / (ms_scan * 1e-3) / 1e9
    print(json.dumps({
        "metric": "n-gram draft proposer: token GB/s", "value": round(nbytes / (ms_step * 1e-3) / 1e9, 2),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32", "data": "synthetic (segments copied from earlier in the sequence or Zipf tokens)",
        "config": {"workload": "ngram-histories", "sequences": n, "tokens": int(tok.size), "n_min": n_min,
                   "n_max": n_max, "k": k},
        "kernel_ms_per_step": {kk: round(v[0] / max(v[1], 1), 4) for kk, v in kern.items() if v[1]},
        "with_drafts": int((cnt > 0).sum().item()),
        "roofline": {"bound": "hbm", "kernel": "ngram_scan", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                     "avg_launch_ms": round(ms_scan, 4), "algorithmic_bytes_per_launch": nbytes}}), flush=True)


def decode_bench(args, torch, spork, synth, runner):
    """A decode loop on one plan: after the workload's step, ``--decode-steps``
    more steps in which every thread appends one token (the host block
    manager), its K/V is written (kv write kernel), the plan is advanced
    (spork_plan_advance: host checks plus one small patch kernel) and the
    step runs. Reports the host time of the appends and the advance against
    the GPU time of the patch and the step, and checks sampled threads of the
    last step against the oracle. The steps are enqueued back to back; the
    host work of step i overlaps the GPU work of earlier steps."""
    import numpy as np

    import oracle
    n = args.decode_steps
    wl = synth.make_named(args.workload, **({"verify_k": args.verify_k} if args.verify_k else {}))
    synth.add_decode_steps(wl, n)
    dw = runner.DeviceWorkload(wl, poison_pool=False)
    step = dw.prepare(0)
    units = step.info["n_units"]
    for _ in range(args.warmup):
        step.run()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    seqs = list(wl.steps[0].seqs)
    ones = [1] * len(seqs)
    # The new tokens' K/V and Q reach the device before the loop (a model's
    # forward pass writes them there); pinned buffers carry each step's slots.
    k_new, v_new, q_new, pinned = [], [], [], []
    for i in range(1, n + 1):
        k_new.append(runner.to_device(np.stack([wl.suffix_k[q][len(wl.suffix_k[q]) - n + i - 1] for q in seqs]),
                                      wl.dtype, dw.device))
        v_new.append(runner.to_device(np.stack([wl.suffix_v[q][len(wl.suffix_v[q]) - n + i - 1] for q in seqs]),
                                      wl.dtype, dw.device))
        q_new.append(runner.to_device(wl.steps[i].q, wl.dtype, dw.device))
        pinned.append(torch.empty(len(seqs), dtype=torch.int64, pin_memory=True))
    torch.cuda.synchronize()
    host_append, host_advance, ev = [], [], []
    for i in range(1, n + 1):
        t0 = time.perf_counter()
        slots, cows = spork.spork_seq_append_batch(dw.cache, seqs, ones)
        t1 = time.perf_counter()
        assert not cows, "a decode append copied a shared block"
        pinned[i - 1].numpy()[:] = slots
        slots_d = pinned[i - 1].to(dw.device, non_blocking=True)
        spork.spork_kv_write(dw.shape, dw.k_pool, dw.v_pool, wl.num_blocks, slots_d, k_new[i - 1], v_new[i - 1],
                             dw.bad_slots)
        step.q.copy_(q_new[i - 1])
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        t2 = time.perf_counter()
        spork.spork_plan_advance(step.plan, dw.cache, step.image)
        t3 = time.perf_counter()
        step.index, step.spec = i, wl.steps[i]
        step.run()
        b.record(stream)
        host_append.append((t1 - t0) * 1e3)
        host_advance.append((t3 - t2) * 1e3)
        ev.append((a, b))
    torch.cuda.synchronize()
    gpu = [a.elapsed_time(b) for a, b in ev]
    info = spork.spork_plan_get_info(step.plan)
    assert info["n_units"] == units and int(dw.bad_slots.item()) == 0
    # oracle parity on sampled threads of the last step
    stl = wl.steps[n]
    starts = np.concatenate([[0], np.cumsum(stl.n_rows)])
    out = step.out.float().cpu().numpy().astype(np.float64)
    worst = 0.0
    pick = sorted({0, len(stl.seqs) // 2, len(stl.seqs) - 1})
    for t in pick:
        seq, r0, nr = stl.seqs[t], int(starts[t]), stl.n_rows[t]
        k, v = wl.context(seq, wl.thread_len(seq, n))
        o, _ = oracle.attend(synth.to_f64(stl.q[r0:r0 + nr], wl.dtype), synth.to_f64(k, wl.dtype),
                             synth.to_f64(v, wl.dtype), wl.sm_scale)
        worst = max(worst, float(np.abs(out[r0:r0 + nr] - o).max()))
    tol = 1e-5 if wl.dtype == synth.F32 else 2e-2
    med = float(np.median(gpu))
    host = float(np.median(np.array(host_append) + np.array(host_advance)))
    print(json.dumps({
        "metric": "decode loop on one plan: host ms per step vs GPU ms per step", "value": round(host / med, 4),
        "unit": "host/GPU time ratio", "n_gpus": 1, "steps": n, "warmup": args.warmup, "ms_per_step": round(med, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == synth.BF16 else "f32", "data": "synthetic (seeded Gaussian K/V/Q)",
        "config": {"workload": wl.name, "decode_steps": n, "threads": len(stl.seqs), "units": units},
        "gpu_ms_per_step": {"median": round(med, 4), "min": round(float(np.min(gpu)), 4),
                            "what": "plan patch kernel + attention step (events)"},
        "host_ms_per_step": {"append_batch_median": round(float(np.median(host_append)), 4),
                             "advance_median": round(float(np.median(host_advance)), 4),
                             "total_median": round(host, 4)},
        "unique_kv_bytes_last_step": info["unique_kv_bytes"],
        "last_step_parity": {"threads": pick, "max_abs": worst, "tol": tol, "ok": worst <= tol}}), flush=True)
    dw.close()
    if worst > tol:
        sys.exit(1)


def cpu_baseline_all(args):
    """The oracle on every benchmark workload with every core, and on the
    two smallest also on one core; one JSON line."""
    import platform

    from paper_2607_03333_amd import synth
    cpu = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), cpu)
    except OSError:
        pass
    res = []
    for i, cfg in enumerate(synth.CONFIGS):
        wl = synth.make(i)
        specs = [(j, st) for j, st in enumerate(wl.steps)]
        for single in ((False, True) if i <= 1 else (False,)):
            r = cpu_baseline(wl, specs, args.cpu_seconds, single_core=single)
            r["workload"] = cfg["name"]
            res.append(r)
            print(f"# {cfg['name']} {'1 core' if single else 'all cores'}: {r['value']:.4f} GB/s ({r['sample']})",
                  file=sys.stderr, flush=True)
        del wl
    print(json.dumps({"metric": "oracle unique-KV GB/s on the host", "cpu": cpu,
                      "logical_cpus": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)),
                      "results": res}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--verify-k", type=int, default=0,
                    help="draft length of the verify workloads (default: the workload's own)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--cpu-baseline-all", action="store_true",
                    help="instead of the benchmark, time the oracle on the host for every workload (all cores, "
                         "and one core for the two smallest) and exit; no GPU is used")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="instead of the benchmark, run one plain device copy of this many MiB "
                         "(reference kernel for the HBM traffic counters) and exit")
    ap.add_argument("--confidence-probes", type=int, default=0,
                    help="instead of the benchmark, time the D2 confidence gate over this many probe "
                         "spans (0..16 positions each) of the 151,936-token vocabulary, bf16 logits")
    ap.add_argument("--decode-steps", type=int, default=0,
                    help="instead of the benchmark, run this many decode steps on one plan after the "
                         "workload's step (spork_plan_advance) and time host against GPU work")
    ap.add_argument("--ngram-seqs", type=int, default=0,
                    help="instead of the benchmark, time the n-gram draft proposer over this many "
                         "token histories of 32768-36864 tokens")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the forked-decode path is "
                                   "measured on a single MI355X; --gpus must be 1"}), flush=True)
        sys.exit(2)

    if args.cpu_baseline_all:
        cpu_baseline_all(args)
        return

    import torch
    from paper_2607_03333_amd import runner, spork, synth

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        sys.exit(1)
    spork.lib()

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20)
        src = torch.empty(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n}), flush=True)
        return

    if args.confidence_probes:
        confidence_bench(args, torch, spork, synth)
        return
    if args.ngram_seqs:
        ngram_bench(args, torch, spork, synth)
        return
    if args.decode_steps:
        decode_bench(args, torch, spork, synth, runner)
        return

    t_gen = time.perf_counter()
    wl = synth.make_named(args.workload, **({"verify_k": args.verify_k} if args.verify_k else {}))
    print(f"# workload {wl.name}: generated in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)

    # Host work of the forks: replay the scenario's block-manager calls alone.
    cache = spork.spork_cache_create(wl.num_blocks, wl.block_size, wl.free_order)
    t_fork = t_other = 0.0
    for st in wl.steps:
        for op in st.ops_before:
            t = time.perf_counter()
            if op[0] == "new":
                spork.spork_seq_new(cache)
                t_other += time.perf_counter() - t
            elif op[0] == "append":
                spork.spork_seq_append(cache, op[1], op[2])
                t_other += time.perf_counter() - t
            elif op[0] == "free":
                spork.spork_seq_free(cache, op[1])
                t_other += time.perf_counter() - t
            else:
                spork.spork_fork(cache, op[1])
                t_fork += time.perf_counter() - t
    shape = spork.make_shape(wl.hq, wl.hkv, wl.d, wl.block_size,
                             spork.SPORK_DTYPE_BF16 if wl.dtype == synth.BF16 else spork.SPORK_DTYPE_F32,
                             wl.sm_scale)
    t = time.perf_counter()
    for st in wl.steps:
        p = spork.spork_plan_create(cache, shape, st.seqs, st.n_rows, st.groups)
        spork.spork_plan_destroy(p)
    t_plan = time.perf_counter() - t
    spork.spork_cache_destroy(cache)
    n_forks = sum(1 for st in wl.steps for op in st.ops_before if op[0] == "fork")

    t_setup = time.perf_counter()
    dw = runner.DeviceWorkload(wl, poison_pool=False)
    steps = dw.prepare_all()
    torch.cuda.synchronize()
    print(f"# device setup {time.perf_counter() - t_setup:.1f} s; units {[s.info['n_units'] for s in steps]} grid {[s.info['attn_grid'] for s in steps]} "
          f"row tiles {[s.info['max_row_tiles'] for s in steps]}", file=sys.stderr, flush=True)

    import numpy as np
    ceiling = read_ceiling(torch, spork)
    print(f"# read ceiling {ceiling['gbps']} GB/s ({ceiling['kernel']})", file=sys.stderr, flush=True)

    def run_step():
        for s in steps:
            s.run()

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()

    # Before every timed step the caches are flushed outside its event pair:
    # a write of a 512 MiB scratch buffer (twice the 256 MB last-level
    # cache), then a read of another 512 MiB buffer, so that the caches hold
    # clean unrelated lines (no write-back of the scratch data lands inside
    # the step) and nothing of the step's inputs.
    stream = torch.cuda.current_stream()
    flush_w = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device="cuda:0")
    flush_r = torch.zeros(FLUSH_BYTES, dtype=torch.uint8, device="cuda:0")
    sink = torch.empty(1024 * 256, dtype=torch.int32, device="cuda:0")

    def flush(i):
        flush_w.fill_(i & 0xFF)
        spork.spork_read_ceiling(flush_r, FLUSH_BYTES, 1024, 0, sink)

    def timed_steps(kernel_events):
        events = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(args.steps)]
        spork.spork_timing_read()
        if kernel_events:
            spork.spork_timing_enable(True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i, (a, b) in enumerate(events):
            if kernel_events:
                spork.spork_timing_enable(False)
                flush(i)
                spork.spork_timing_enable(True)
            else:
                flush(i)
            a.record(stream)
            run_step()
            b.record(stream)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        spork.spork_timing_enable(False)
        kern = spork.spork_timing_read()
        return np.array([a.elapsed_time(b) for a, b in events]), dt, kern

    # The timed region: K steps, each timed alone by HIP events on its stream.
    step_ms, wall, _ = timed_steps(False)
    ms_step = float(np.median(step_ms))
    # Per-kernel durations: the same protocol again with the library's events
    # around each of its launches (they add a few microseconds per launch to
    # the step, so the step times above are taken without them).
    _, _, kern = timed_steps(True)
    # The same steps back to back (no flush), as a separate figure.
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(args.steps):
        run_step()
    end.record(stream)
    torch.cuda.synchronize()
    ms_back_to_back = start.elapsed_time(end) / args.steps
    del flush_w, flush_r, sink

    unique = sum(s.info["unique_kv_bytes"] for s in steps)
    flat = sum(s.info["flat_kv_bytes"] for s in steps)
    verified = 0
    drafts_checked = 0
    for s in steps:
        if s.verify:
            verified += int((s.accept_len.cpu() + 1).sum().item())
            drafts_checked += s.n_verify * s.spec.verify_k
    value = unique / (ms_step * 1e-3) / 1e9

    attn_ms, attn_n = kern["attn_partial"]
    attn_avg_ms = attn_ms / max(attn_n, 1)
    logits_bytes = sum(s.logits.numel() * s.logits.element_size() for s in steps if s.verify)
    # With the persistent bf16 kernel the verify step's argmax runs inside the
    # attention launch (no argmax launch is timed): its logits count there.
    fused_logits = logits_bytes if kern["argmax"][1] == 0 else 0
    attn_bytes_per_launch = (unique + fused_logits) / len(steps)
    achieved = attn_bytes_per_launch / (attn_avg_ms * 1e-3) / 1e9
    traffic = measured_traffic(wl.name)
    flops_per_launch = sum(attention_flops(wl, s.index, s.spec) for s in steps) / len(steps)
    dt = "bf16" if wl.dtype == synth.BF16 else "f32"
    intensity = flops_per_launch / attn_bytes_per_launch
    ridge = MFMA_PEAK_TFLOPS[dt] * 1e12 / (HBM_PEAK_GBPS * 1e9)
    if intensity > ridge:
        # past the ridge point the launch is priced against the matrix cores
        tflops = flops_per_launch / (attn_avg_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "kernel": "attn_partial", "achieved": round(tflops, 1),
                "peak": MFMA_PEAK_TFLOPS[dt], "unit": "TFLOP/s", "frac": round(tflops / MFMA_PEAK_TFLOPS[dt], 4),
                "traffic": traffic}
    else:
        roof = {"bound": "hbm", "kernel": "attn_partial", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "traffic": traffic}
    roof.update({
        "pct_of_ceiling": round(100.0 * achieved / ceiling["gbps"], 2),
        "avg_launch_ms": round(attn_avg_ms, 4),
        "algorithmic_bytes_per_launch": attn_bytes_per_launch,
        "algorithmic_bytes": "unique KV" + (" + verify logits (argmax inside the launch)" if fused_logits else ""),
        "hbm_gbps": round(achieved, 1),
        "algorithmic_flops_per_launch": flops_per_launch,
        "tflops": round(flops_per_launch / (attn_avg_ms * 1e-3) / 1e12, 1),
        "intensity_flop_per_byte": round(intensity, 1),
        "ridge_flop_per_byte": round(ridge, 1),
    })

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic (seeded Gaussian K/V/Q" + (", planted greedy logits)" if logits_bytes else ")"),
        "config": {
            "workload": wl.name, "query_heads": wl.hq, "kv_heads": wl.hkv, "head_dim": wl.d,
            "block_size": wl.block_size, "sessions": len(wl.prefix_len),
            "threads": sum(len(s.spec.seqs) for s in steps),
            "query_rows": sum(sum(s.spec.n_rows) for s in steps),
            "shared_prefix_tokens": wl.prefix_len[0], "verify_k": max(s.spec.verify_k for s in steps),
            "parallelism": "single GPU",
        },
        "pct_of_8TBps": round(100.0 * value / HBM_PEAK_GBPS, 2),
        "pct_of_ceiling": round(100.0 * value / ceiling["gbps"], 2),
        "timing": {"protocol": "before each timed step (outside its events) a 512 MiB scratch write, then a "
                               "512 MiB read of another buffer; per-step HIP events; value and ms_per_step "
                               "from the median step; per-kernel times from a second pass",
                   "ms_per_step_median": round(ms_step, 4), "ms_per_step_min": round(float(step_ms.min()), 4),
                   "ms_per_step_mean": round(float(step_ms.mean()), 4),
                   "ms_per_step_back_to_back": round(ms_back_to_back, 4),
                   "value_back_to_back": round(unique / (ms_back_to_back * 1e-3) / 1e9, 2)},
        "read_ceiling": ceiling,
        "verified_tokens_per_s": round(verified / (ms_step * 1e-3), 1) if verified else None,
        "drafts_checked_per_s": round(drafts_checked / (ms_step * 1e-3), 1) if drafts_checked else None,
        "unique_kv_bytes_per_step": unique,
        "logits_bytes_per_step": logits_bytes,
        "flat_kv_bytes_per_step": flat,
        "kernel_ms_per_step": {k: round(v[0] / args.steps, 4) for k, v in kern.items() if v[1]},
        "host_ms": {"forks": round(t_fork * 1e3, 3), "n_forks": n_forks, "appends_and_new": round(t_other * 1e3, 3),
                    "plan": round(t_plan * 1e3, 3)},
        "wall_s_timed_region": round(wall, 4),
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, [(s.index, s.spec) for s in steps], args.cpu_seconds)
    dw.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
