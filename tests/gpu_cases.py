"""Shared helpers of the GPU parity tests: run a workload through the C ABI,
compute the oracle on the same logical inputs, compare."""
import sys

import numpy as np
import torch

import oracle
from paper_2607_03333_amd import runner, synth

FP32_TOL = 1e-5     # max-abs on fp32 outputs
BF16_TOL = 2e-2     # max-abs on bf16 outputs
BF16_RMS = 1e-2     # relative RMS error gate on bf16 outputs
LSE_REL = 1e-3      # lse relative error gate


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def thread_len(wl, step_index, seq):
    return wl.thread_len(seq, step_index)


def oracle_rows(wl, step_index, pick=None):
    """Oracle (o, lse) for the threads of a step (all, or the indices in ``pick``)."""
    st = wl.steps[step_index]
    res = {}
    row = 0
    for t, (seq, n) in enumerate(zip(st.seqs, st.n_rows)):
        if pick is None or t in pick:
            L = wl.thread_len(seq, step_index)
            k, v = wl.context(seq, L)
            q = synth.to_f64(st.q[row:row + n], wl.dtype)
            o, lse = oracle.attend(q, synth.to_f64(k, wl.dtype), synth.to_f64(v, wl.dtype), wl.sm_scale)
            res[t] = (row, o, lse)
        row += n
    return res


def compare_attention(wl, step, pick=None, tag="", ref=None):
    """Element-wise comparison of a step's GPU output with the oracle
    (``ref``: precomputed {thread: (first row, o, lse)}, else computed here)."""
    if ref is None:
        ref = oracle_rows(wl, step.index, pick)
    out = step.out.float().cpu().numpy().astype(np.float64)
    lse = step.lse.cpu().numpy().astype(np.float64)
    worst = 0.0
    err2 = 0.0
    ref2 = 0.0
    lse_worst = 0.0
    for t, (row, o, l) in ref.items():
        n = o.shape[0]
        got = out[row:row + n]
        assert np.all(np.isfinite(got)), f"{tag}: non-finite output for thread {t}"
        worst = max(worst, float(np.max(np.abs(got - o))))
        err2 += float(np.sum((got - o) ** 2))
        ref2 += float(np.sum(o ** 2))
        lse_worst = max(lse_worst, float(np.max(np.abs(lse[row:row + n] - l) / np.maximum(1.0, np.abs(l)))))
    tol = FP32_TOL if wl.dtype == "f32" else BF16_TOL
    rel_rms = (err2 / max(ref2, 1e-300)) ** 0.5
    say(f"  {tag}: {len(ref)} threads, max-abs {worst:.3e} (tol {tol:g}) rel-rms {rel_rms:.3e} lse-rel {lse_worst:.3e}")
    assert worst <= tol, f"{tag}: max-abs error {worst} > {tol}"
    if wl.dtype != "f32":
        assert rel_rms <= BF16_RMS, f"{tag}: relative RMS error {rel_rms}"
    assert lse_worst <= LSE_REL, f"{tag}: lse relative error {lse_worst}"
    return worst


def compare_accept(wl, step, tag=""):
    st = step.spec
    logits = synth.to_f64(st.logits, wl.logits_dtype)
    g = oracle.argmax_rows(logits)
    a, n = oracle.accept_drafts(g, st.drafts)
    got_g = step.argmax.cpu().numpy()
    got_a = step.accept_len.cpu().numpy()
    got_n = step.next_token.cpu().numpy()
    assert np.array_equal(got_g, g), f"{tag}: argmax differs at rows {np.nonzero(got_g != g)[0][:10]}"
    assert np.array_equal(got_a, a), f"{tag}: accept lengths differ"
    assert np.array_equal(got_n, n), f"{tag}: next tokens differ"
    assert np.array_equal(got_a, st.planted_accept) and np.array_equal(got_n, st.planted_next)
    say(f"  {tag}: accept {got_a.tolist()[:12]} bit-exact vs oracle and planted values")


def compare_tables(wl, dw):
    """Block tables, refcounts and free queue of the library vs the oracle manager."""
    from paper_2607_03333_amd import spork
    bm = oracle.BlockManager(wl.num_blocks, wl.block_size, wl.free_order)
    for st in wl.steps:
        for op in st.ops_before:
            if op[0] == "new":
                bm.seq_new()
            elif op[0] == "append":
                bm.append(op[1], op[2])
            elif op[0] == "free":
                bm.free_seq(op[1])
            else:
                bm.fork(op[1])
    for s in bm.tables:
        assert spork.spork_block_table(dw.cache, s).tolist() == bm.table(s)
    assert spork.spork_free_blocks(dw.cache).tolist() == bm.free_list()


def snapshot(step):
    """Copies of everything a step writes."""
    got = [step.out.clone(), step.lse.clone()]
    if step.verify:
        got += [step.argmax.clone(), step.accept_len.clone(), step.next_token.clone()]
    return got


def assert_bit_equal(first, step, tag):
    """A second run of a step reproduces the first bit for bit: units write
    fixed partial slots and every output's partials merge in a fixed order,
    whichever workgroup runs a unit or merges an output."""
    again = snapshot(step)
    names = ["out", "lse", "argmax", "accept_len", "next_token"]
    for name, x, y in zip(names, first, again):
        assert torch.equal(x, y), f"{tag}: {name} differs between two runs"
    say(f"  {tag}: second run bit-identical")


def run_workload(wl, tag, pick=None, check_tables=True, repeat_check=True):
    """Run every step through the C ABI right after preparing it (before the
    next step's appends, which may reuse freed blocks) and compare it with
    the oracle; optionally run it again and require bit-identical results."""
    dw = runner.DeviceWorkload(wl)
    try:
        for i in range(len(wl.steps)):
            step = dw.prepare(i)
            assert int(dw.bad_slots.item()) == 0
            say(f"[{tag}] step {step.index}: threads {len(step.spec.seqs)} rows {sum(step.spec.n_rows)} "
                f"units {step.info['n_units']} grid {step.info['attn_grid']} row_tiles {step.info['max_row_tiles']}")
            step.poison()
            step.run()
            torch.cuda.synchronize()
            compare_attention(wl, step, pick, tag=f"{tag} step {step.index}")
            if step.verify:
                compare_accept(wl, step, tag=f"{tag} step {step.index}")
            if repeat_check:
                first = snapshot(step)
                step.poison()
                step.run()
                torch.cuda.synchronize()
                assert_bit_equal(first, step, f"{tag} step {step.index}")
        if check_tables:
            compare_tables(wl, dw)
        return dw
    except Exception:
        dw.close()
        raise
