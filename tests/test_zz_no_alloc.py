"""spork_verify_accept_noalloc (the library's per-device scratch array in
place of a caller workspace) against spork_verify_accept on the same
inputs, bit for bit: a mixed decode + verify step, then a smaller decode
step right after it (the scratch keeps the first call's contents), then the
larger step again (its control words must be cleared again), and an
accept-only call. Every result of the no-allocation path must equal the
workspace path's, which the parity tests check against the oracle."""
import pytest
import torch

from gpu_cases import compare_accept, compare_attention, say
from paper_2607_03333_amd import runner, spork, synth

pytestmark = pytest.mark.gpu


def _noalloc(step, dw):
    """Run the step through the no-allocation entry point into fresh
    NaN/-1 outputs; returns them."""
    out = torch.full_like(step.out, float("nan"))
    lse = torch.full_like(step.lse, float("nan"))
    res = {"out": out, "lse": lse}
    if step.verify:
        res.update(accept_len=torch.full_like(step.accept_len, -1), next_token=torch.full_like(step.next_token, -1),
                   argmax=torch.full_like(step.argmax, -1))
        spork.spork_verify_accept_noalloc(step.plan, step.image, step.q, dw.k_pool, dw.v_pool, out, lse, step.logits,
                                          runner._SPORK_DTYPE[dw.wl.logits_dtype], step.vocab, step.drafts,
                                          step.n_verify, step.spec.verify_k, res["accept_len"], res["next_token"],
                                          res["argmax"])
    else:
        spork.spork_verify_accept_noalloc(step.plan, step.image, step.q, dw.k_pool, dw.v_pool, out, lse, None,
                                          spork.SPORK_DTYPE_BF16, 1, None, 0, 0, None, None, None)
    return res


def _same(step, res, tag):
    assert torch.equal(res["out"], step.out), f"{tag}: out differs"
    assert torch.equal(res["lse"], step.lse), f"{tag}: lse differs"
    if step.verify:
        for name in ("accept_len", "next_token", "argmax"):
            assert torch.equal(res[name], getattr(step, name)), f"{tag}: {name} differs"
    say(f"  {tag}: no-allocation results equal the workspace path's bit for bit")


def test_noalloc_matches_the_workspace_path():
    big = synth.make(4, sessions=4, prefix=1500, suffix=("loguniform", 1, 400), vocab=3000)
    small = synth.make(2, sessions=2, prefix=600, suffix=("uniform", 1, 120))
    dws = [runner.DeviceWorkload(big), runner.DeviceWorkload(small)]
    try:
        s_big, s_small = dws[0].prepare_all()[-1], dws[1].prepare_all()[-1]
        assert s_big.info["workspace_bytes"] > s_small.info["workspace_bytes"]
        assert s_big.info["control_bytes"] >= s_small.info["control_bytes"]
        say(f"[noalloc] big step: {s_big.info['workspace_bytes']} workspace bytes; small: "
            f"{s_small.info['workspace_bytes']}")
        for s in (s_big, s_small):       # references through the caller-workspace entry point
            s.poison()
            s.run()
        torch.cuda.synchronize()
        compare_attention(big, s_big, tag="noalloc reference big")
        compare_accept(big, s_big, tag="noalloc reference big")
        compare_attention(small, s_small, tag="noalloc reference small")
        r1 = _noalloc(s_big, dws[0])
        r2 = _noalloc(s_small, dws[1])    # the second call, smaller, right after the first
        r3 = _noalloc(s_big, dws[0])      # larger again
        torch.cuda.synchronize()
        _same(s_big, r1, "big step (first call)")
        _same(s_small, r2, "small step (second call)")
        _same(s_big, r3, "big step (third call)")
        # accept only (no plan)
        acc = torch.full_like(s_big.accept_len, -1)
        nxt = torch.full_like(s_big.next_token, -1)
        spork.spork_verify_accept_noalloc(None, None, None, None, None, None, None, s_big.logits,
                                          spork.SPORK_DTYPE_BF16, s_big.vocab, s_big.drafts, s_big.n_verify,
                                          s_big.spec.verify_k, acc, nxt, None)
        torch.cuda.synchronize()
        assert torch.equal(acc, s_big.accept_len) and torch.equal(nxt, s_big.next_token)
        say("  accept-only call: equal")
    finally:
        for dw in dws:
            dw.close()
