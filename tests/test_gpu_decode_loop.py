"""A decode loop reusing one plan (spork_plan_advance): every thread appends
one token per step, the plan's device image is patched, and each step is
compared with the oracle on every thread (accept bit-exactly on verify
steps). Steps cross block boundaries, so the patches carry new table
entries as well as the grown private ranges."""
import pytest
import torch

from gpu_cases import compare_accept, compare_attention, say
from paper_2607_03333_amd import runner, synth

pytestmark = pytest.mark.gpu


def _run_loop(wl, base, n_steps, tag):
    synth.add_decode_steps(wl, n_steps)
    dw = runner.DeviceWorkload(wl)
    try:
        for i in range(base + 1):
            step = dw.prepare(i)
        units = step.info["n_units"]
        for i in range(base, base + n_steps + 1):
            if i > base:
                dw.advance(step, i)
                assert step.info["n_units"] == units, "the plan was not reused"
            assert int(dw.bad_slots.item()) == 0
            step.poison()
            step.run()
            torch.cuda.synchronize()
            if i == base or (i - base) % 8 == 0 or i == base + n_steps:
                compare_attention(wl, step, tag=f"{tag} step {i}")
                if step.verify:
                    compare_accept(wl, step, tag=f"{tag} step {i}")
        say(f"[{tag}] {n_steps} decode steps on one plan of {units} units")
    finally:
        dw.close()


@pytest.mark.parametrize("name,kw,n_steps", [
    ("qwen3-30b-a3b-mixed", dict(sessions=3, prefix=1000, suffix=("loguniform", 1, 300), vocab=3000), 40),
    ("qwen3-32b-decode", dict(sessions=2, prefix=700, suffix=("uniform", 1, 200)), 40),
    ("qwen3-4b-decode", dict(sessions=2, prefix=512, suffix=("uniform", 1, 64), block_size=32), 40),
    ("tiny-fork-f32", {}, 24),
], ids=["mixed", "32b-decode", "4b-decode-bs32", "tiny-f32"])
def test_decode_loop_reuses_the_plan(name, kw, n_steps):
    wl = synth.make(name, **kw)
    _run_loop(wl, len(wl.steps) - 1, n_steps, f"loop {name}")


def test_decode_loop_on_a_fork_tree():
    wl = synth.make_tree(sessions=2, prefix=600, stride=40, probes=3, probe_tokens=(1, 20), main_extra=(1, 40))
    _run_loop(wl, 0, 24, "loop tree")
