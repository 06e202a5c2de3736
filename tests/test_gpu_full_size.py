"""GPU parity at the workloads' full sizes, in the configuration bench.py times.

The whole batch runs through the C ABI; the oracle recomputes a sample of
threads one by one (the first and last thread, the longest context, the
shortest private range, a verify thread where there is one, and for the
staggered fork tree and the probe prefill every thread of the first and last
session), element by element. Argmax and accept are compared on every row, bit-exactly, against
the oracle and against the generator's planted values. Every output is also
checked by a second run: which workgroup computes which chunk of a unit
changes from run to run, so a chunk lost or counted twice anywhere in the
batch shows up as a difference between the runs (they may differ only by
fp32 summation order).
"""
import numpy as np
import pytest
import torch

from paper_2607_03333_amd import runner, synth
from gpu_cases import BF16_TOL, FP32_TOL, LSE_REL, compare_accept, compare_attention, say

pytestmark = pytest.mark.gpu


def _pick(wl, step_index):
    st = wl.steps[step_index]
    n = len(st.seqs)
    lens = [wl.thread_len(s, step_index) for s in st.seqs]
    priv = [L - wl.prefix_len[next(t.session for t in wl.threads if t.seq == s)] for s, L in zip(st.seqs, lens)]
    pick = {0, n // 2, n - 1, int(np.argmax(lens)), int(np.argmin(priv))}
    verify = [i for i, r in enumerate(st.n_rows) if r > 1]
    if verify:
        pick.add(verify[-1])
    if wl.name in (synth.TREE_NAME, synth.PREFILL_NAME):
        # every thread of the first and the last session: each level of both trees
        sess = [wl.thread(q).session for q in st.seqs]
        pick |= {i for i, x in enumerate(sess) if x in (sess[0], sess[-1])}
    return sorted(pick)


@pytest.mark.parametrize("index,over", [(0, {}), (1, {}), (2, {}), (3, {}), (4, {}), (synth.TREE_NAME, {}),
                                        (synth.PREFILL_NAME, {}), ("qwen3-32b-verify", dict(verify_k=50)),
                                        ("supersede", {})],
                         ids=["0", "1", "2", "3", "4", "tree", "prefill", "verify-k50", "tree-supersede"])
def test_full_size_workload(index, over):
    if index == "supersede":
        wl = synth.add_supersession_step(synth.make_tree())
    else:
        wl = synth.make_named(index, **over)
    say(f"[full {wl.name}] generated; blocks {wl.num_blocks}")
    dw = runner.DeviceWorkload(wl, poison_pool=True)
    try:
        steps = dw.prepare_all()
        assert int(dw.bad_slots.item()) == 0
        for step in steps:
            step.poison()
            step.run()
            torch.cuda.synchronize()
            pick = _pick(wl, step.index)
            say(f"[full {wl.name}] step {step.index}: {step.info['n_units']} units on {step.info['attn_grid']} workgroups, checking threads {pick}")
            compare_attention(wl, step, set(pick), tag=f"full {wl.name} step {step.index}")
            out = step.out.float().clone()
            lse = step.lse.clone()
            assert bool(torch.isfinite(out).all()), "non-finite outputs"
            if step.verify:
                compare_accept(wl, step, tag=f"full {wl.name} step {step.index}")
            step.poison()
            step.run()
            torch.cuda.synchronize()
            tol = FP32_TOL if step.out.dtype == torch.float32 else BF16_TOL
            d_out = float((out - step.out.float()).abs().max())
            d_lse = float(((lse - step.lse).abs() / lse.abs().clamp_min(1.0)).max())
            say(f"  full {wl.name} step {step.index}: all {out.shape[0]} x {out.shape[1]} outputs, run vs run: "
                f"max-abs {d_out:.3e} lse-rel {d_lse:.3e}")
            assert d_out <= tol and d_lse <= LSE_REL
    finally:
        dw.close()
