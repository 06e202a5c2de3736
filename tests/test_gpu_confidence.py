"""GPU parity of the D2 confidence gate (Section 4.2) against the oracle.

Through the C ABI: spork_probe_confidence on seeded probe logits (bf16 and
float32, the Qwen3 vocabulary of 151,936 and ragged small vocabularies) is
compared with oracle.top1_logprob / span_confidence / confidence_gate in
float64.

Tolerances: greedy tokens bit-exact. The kernel sums the exponentials in
float32: each term carries at most a few ulp of relative error (the exponent
argument's rounding and the hardware exp2), and a thread adds at most a few
hundred terms in order before a tree combine of about twenty levels, so the
relative error of the sum, which is the absolute error of the log-probability,
stays below 4e-5 in the worst case (about 1e-6 in practice); the gate allows
1e-4. The gate's decision is taken in float32 on the kernel side; where the
oracle's score is within 1e-4 of theta, the decision is checked against the
kernel's own score instead.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_03333_amd import runner, spork, synth
from gpu_cases import say

pytestmark = pytest.mark.gpu

THETA = 0.90
LOGPROB_TOL = 1e-4
_DT = {synth.BF16: spork.SPORK_DTYPE_BF16, synth.F32: spork.SPORK_DTYPE_F32}


def run_confidence(logits, dtype, span_off, theta=THETA, n_rows=None):
    dev = torch.device("cuda:0")
    n_rows = logits.shape[0] if n_rows is None else n_rows
    vocab = logits.shape[1]
    n_probes = len(span_off) - 1
    x = runner.to_device(logits, dtype, dev) if logits.size else None
    off = torch.tensor(np.asarray(span_off, dtype=np.int32), device=dev)
    am = torch.full((max(n_rows, 1),), -7, dtype=torch.int32, device=dev)
    lp = torch.full((max(n_rows, 1),), float("nan"), dtype=torch.float32, device=dev)
    conf = torch.full((max(n_probes, 1),), float("nan"), dtype=torch.float32, device=dev)
    commit = torch.full((max(n_probes, 1),), -7, dtype=torch.int32, device=dev)
    ws = torch.empty(max(spork.spork_confidence_workspace_bytes(n_rows, vocab), 1), dtype=torch.uint8, device=dev)
    ws.fill_(0xA5)  # any contents on entry
    spork.spork_probe_confidence(x, _DT[dtype], vocab, n_rows, off, n_probes, theta, am, lp, conf, commit, ws)
    torch.cuda.synchronize()
    return (am.cpu().numpy()[:n_rows], lp.cpu().numpy()[:n_rows].astype(np.float64),
            conf.cpu().numpy()[:n_probes].astype(np.float64), commit.cpu().numpy()[:n_probes])


def check(logits, dtype, span_off, theta=THETA, tag=""):
    am, lp, conf, commit = run_confidence(logits, dtype, span_off, theta)
    x = synth.to_f64(logits, dtype)
    want_l = oracle.top1_logprob(x)
    want_c = oracle.span_confidence(want_l, span_off)
    want_g = oracle.confidence_gate(want_c, theta)
    err_l = float(np.max(np.abs(lp - want_l))) if len(lp) else 0.0
    err_c = float(np.max(np.abs(conf - want_c))) if len(conf) else 0.0
    say(f"  {tag}: rows {x.shape[0]} vocab {x.shape[1]} probes {len(span_off) - 1} "
        f"max|dl| {err_l:.2e} max|dc| {err_c:.2e} commits {int(commit.sum())}")
    assert np.array_equal(am, oracle.argmax_rows(x))
    assert err_l <= LOGPROB_TOL and err_c <= LOGPROB_TOL
    far = np.abs(want_c - theta) > LOGPROB_TOL
    assert np.array_equal(commit[far].astype(bool), want_g[far])
    assert np.array_equal(commit.astype(bool), conf.astype(np.float32) >= np.float32(theta))
    return am, lp, conf, commit


@pytest.mark.parametrize("dtype", [synth.BF16, synth.F32])
@pytest.mark.parametrize("vocab,n_probes", [(151936, 24), (1003, 40), (4096, 300), (7, 9)])
def test_confidence_matches_oracle(dtype, vocab, n_probes):
    say(f"confidence parity dtype={dtype} vocab={vocab} probes={n_probes}")
    b = synth.probe_batch(n_probes, vocab, dtype=dtype, seed=vocab + n_probes)
    check(b.logits, dtype, b.span_off, tag=f"{dtype} V={vocab}")


def test_confidence_full_size_many_probes():
    # 256 probes with spans up to 16 tokens: several thousand rows of the
    # Qwen3 vocabulary (one chunk per row)
    say("confidence full size: 256 probes, spans 0..16, vocab 151936, bf16")
    b = synth.probe_batch(256, 151936, span=(0, 16), seed=7)
    check(b.logits, synth.BF16, b.span_off, tag="full")


def test_masked_entries_and_ties():
    say("confidence with -inf entries and planted ties")
    b = synth.probe_batch(30, 2048, dtype=synth.F32, seed=3, tie_prob=0.5, neg_inf_prob=0.3)
    check(b.logits, synth.F32, b.span_off, tag="masked")
    # a row with two tied maxima far above the rest: l = -ln 2, lowest index wins
    x = np.full((3, 300), -30.0, dtype=np.float32)
    x[:, 17] = x[:, 250] = 5.0
    am, lp, conf, commit = check(x, synth.F32, [0, 3], tag="tie")
    assert am.tolist() == [17, 17, 17] and abs(conf[0] - 0.5) < 1e-6 and commit[0] == 0


def test_empty_short_and_out_of_range_spans():
    say("confidence edge spans")
    b = synth.probe_batch(6, 512, dtype=synth.F32, seed=11, span=(3, 3))
    n = b.logits.shape[0]
    # empty, single-row, reversed and out-of-range spans: clamped, score 1
    off = np.array([0, 0, 1, 1, n], dtype=np.int32)
    check(b.logits, synth.F32, off, tag="edges")
    _, _, conf, commit = run_confidence(b.logits, synth.F32, np.array([5, 2, n + 40, -3], dtype=np.int32))
    x = synth.to_f64(b.logits, synth.F32)
    l = oracle.top1_logprob(x)
    # [5, 2) reversed -> empty; [2, n + 40) clamped to [2, n); [n + 40, -3) clamped to [n, 0), reversed -> empty
    want = oracle.span_confidence(l, [5, 5, 2, n, n])[[0, 2, 3]]
    assert np.allclose(conf, want, rtol=0, atol=LOGPROB_TOL)
    assert conf[0] == 1.0 and conf[2] == 1.0 and commit[0] == 1 and commit[2] == 1
    # no rows at all: every probe scores 1 and commits
    _, _, conf, commit = run_confidence(np.zeros((0, 100), np.float32), synth.F32, [0, 0, 0], n_rows=0)
    assert conf.tolist() == [1.0, 1.0] and commit.tolist() == [1, 1]


def test_theta_edges():
    say("confidence gate at theta 0 and above 1")
    b = synth.probe_batch(20, 999, dtype=synth.BF16, seed=5)
    _, _, _, commit = check(b.logits, synth.BF16, b.span_off, theta=0.0, tag="theta0")
    assert commit.all()
    _, _, conf, commit = check(b.logits, synth.BF16, b.span_off, theta=1.0000001, tag="theta>1")
    assert not commit.any()
