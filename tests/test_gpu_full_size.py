"""GPU parity at the workloads' full sizes, in the launch configuration
bench.py times.

Every thread of every step of the five benchmark workloads and of the fork
tree (with its supersession step) is compared with the oracle element by
element; for the probe prefill (about 60 query rows per session) every
thread of 16 of the 64 sessions. The oracle runs in worker processes on the
host's cores (each rebuilds the workload from its seeds and draws the K/V of
its threads) while the GPU runs. Argmax and accept are compared bit-exactly on every row, against the
oracle and against the generator's planted values. Each step then runs a
second time from poisoned outputs and workspace and must reproduce the first
run bit for bit. Steps run right after they are prepared, before the next
step's appends; in the supersession case the pool is shrunk so that the
second step's appends reuse the blocks its free returned (stale KV).
"""
import numpy as np
import pytest
import torch

import oracle_pool
from gpu_cases import compare_accept, compare_attention, say, snapshot, assert_bit_equal
from paper_2607_03333_amd import runner, synth

pytestmark = pytest.mark.gpu

CASES = {
    "0": (synth.CONFIGS[0]["name"], {}, False),
    "1": (synth.CONFIGS[1]["name"], {}, False),
    "2": (synth.CONFIGS[2]["name"], {}, False),
    "3": (synth.CONFIGS[3]["name"], {}, False),
    "4": (synth.CONFIGS[4]["name"], {}, False),
    "tree": (synth.TREE_NAME, {}, False),
    "prefill": (synth.PREFILL_NAME, {}, False),
    "verify-k50": ("qwen3-32b-verify", {"verify_k": 50}, False),
    "tree-supersede": (synth.TREE_NAME, {}, True),
}


@pytest.fixture(scope="module")
def pool():
    p = oracle_pool.OraclePool()
    yield p
    p.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("case_id", list(CASES))
def test_full_size_workload(case_id, pool):
    case = CASES[case_id]
    name, kw, supersede = case
    wl = synth.make_named(name, **kw)
    if supersede:
        synth.add_supersession_step(wl)
        oracle_pool.tight_pool(wl)
        reused = oracle_pool.reused_blocks(wl)
        assert reused, "the supersession step must reuse freed blocks"
        say(f"[full {wl.name}] pool of {wl.num_blocks} blocks; step 1 reuses {len(reused)} freed blocks")
    say(f"[full {wl.name}] generated; blocks {wl.num_blocks}")
    dw = runner.DeviceWorkload(wl, poison_pool=True)
    try:
        sessions = None
        if case_id == "prefill":
            n_sess = len(wl.prefix_len)
            sessions = {int(x) for x in np.linspace(0, n_sess - 1, 16)}
        for i in range(len(wl.steps)):
            futures = pool.submit(case, wl, i, sessions)
            step = dw.prepare(i)
            assert int(dw.bad_slots.item()) == 0
            tag = f"full {wl.name} step {i}"
            say(f"[{tag}] {len(step.spec.seqs)} threads, {step.info['n_units']} units on "
                f"{step.info['attn_grid']} workgroups of {step.info['attn_waves']} waves")
            step.poison()
            step.run()
            torch.cuda.synchronize()
            first = snapshot(step)
            assert bool(torch.isfinite(step.out.float()).all()), "non-finite outputs"
            if step.verify:
                compare_accept(wl, step, tag=tag)
            step.poison()
            step.run()
            torch.cuda.synchronize()
            assert_bit_equal(first, step, tag)
            ref = {}
            for n_done, f in enumerate(futures, 1):
                for t, row, o, lse in f.result():
                    ref[t] = (row, o, lse)
                if n_done % 16 == 0 or n_done == len(futures):
                    say(f"  {tag}: oracle {n_done}/{len(futures)} sessions")
            if sessions is None:
                assert sorted(ref) == list(range(len(step.spec.seqs)))
            compare_attention(wl, step, tag=tag, ref=ref)
    finally:
        dw.close()


@pytest.mark.timeout(900)
def test_full_size_decode_loop(pool):
    """The bench workload, then 16 decode steps on one plan (every thread
    appends a token per step; spork_plan_advance patches the image): every
    thread of the last step against the oracle, and that step run twice bit
    for bit."""
    case = ("qwen3-30b-a3b-mixed", {}, False)
    wl = synth.make_named(case[0])
    synth.add_decode_steps(wl, 16)
    dw = runner.DeviceWorkload(wl, poison_pool=True)
    try:
        step = dw.prepare(0)
        units = step.info["n_units"]
        for i in range(1, len(wl.steps)):
            dw.advance(step, i)
            step.run()
        torch.cuda.synchronize()
        assert step.info["n_units"] == units and int(dw.bad_slots.item()) == 0
        last = len(wl.steps) - 1
        futures = pool.submit(oracle_pool.decode_case(case, 16), wl, last)
        tag = f"full decode loop step {last}"
        step.poison()
        step.run()
        torch.cuda.synchronize()
        first = snapshot(step)
        compare_accept(wl, step, tag=tag)
        step.poison()
        step.run()
        torch.cuda.synchronize()
        assert_bit_equal(first, step, tag)
        ref = {t: (row, o, lse) for f in futures for t, row, o, lse in f.result()}
        assert sorted(ref) == list(range(len(step.spec.seqs)))
        compare_attention(wl, step, tag=tag, ref=ref)
    finally:
        dw.close()
