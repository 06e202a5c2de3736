"""Pins for the oracle top-1 log-probability and D2 confidence gate (Section 4.2).

References: scipy.special.logsumexp (an implementation independent of the
oracle's), torch.softmax in float64, closed forms for equal, tied and dominant
logits, a hand-worked span trace, and a brute-force span scan.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

from oracle import top1_logprob, span_confidence, confidence_gate

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_trace():
    with open(os.path.join(GOLDEN, "confidence_trace.json")) as f:
        g = json.load(f)
    x = np.array(g["logits"])
    l = top1_logprob(x)
    assert np.allclose(np.exp(l), g["expect_top1_prob"], rtol=0, atol=1e-12)
    assert np.argmax(x, axis=1).tolist() == g["expect_argmax"]
    s = span_confidence(l, g["span_off"])
    assert np.allclose(s, g["expect_score"], rtol=0, atol=1e-12)
    assert confidence_gate(s, g["theta"]).tolist() == g["expect_commit"]


def test_matches_scipy_logsumexp():
    rng = np.random.default_rng(31)
    x = rng.standard_normal((64, 1000)) * 4.0
    want = x.max(axis=1) - logsumexp(x, axis=1)
    assert np.allclose(top1_logprob(x), want, rtol=0, atol=1e-12)


def test_matches_torch_softmax_of_argmax():
    rng = np.random.default_rng(32)
    x = rng.standard_normal((16, 151936)).astype(np.float32) * 3.0
    p = torch.softmax(torch.from_numpy(x).double(), dim=1).max(dim=1).values.numpy()
    assert np.allclose(np.exp(top1_logprob(x)), p, rtol=1e-12, atol=0)


@pytest.mark.parametrize("v", [1, 2, 7, 151936])
def test_closed_forms(v):
    # equal logits: uniform distribution
    assert top1_logprob(np.full((1, v), 3.5))[0] == pytest.approx(-math.log(v), abs=1e-12)
    if v >= 3:
        # two tied maxima far above the rest
        x = np.full((1, v), -1e4)
        x[0, 0] = x[0, v - 1] = 2.0
        assert top1_logprob(x)[0] == pytest.approx(-math.log(2.0), abs=1e-12)
    # one maximum d above v - 1 equal others
    d = 5.0
    x = np.zeros((1, v))
    x[0, v // 2] = d
    assert top1_logprob(x)[0] == pytest.approx(-math.log1p((v - 1) * math.exp(-d)), abs=1e-12)


def test_shift_invariance_and_bounds():
    rng = np.random.default_rng(33)
    x = rng.standard_normal((20, 300))
    l = top1_logprob(x)
    assert np.allclose(top1_logprob(x + 1234.5), l, atol=1e-9)
    assert np.all(l <= 0) and np.all(l >= -math.log(300) - 1e-12)


def test_span_brute_force():
    rng = np.random.default_rng(34)
    for _ in range(100):
        n = int(rng.integers(1, 6))
        lens = rng.integers(0, 6, size=n)
        off = np.concatenate([[0], np.cumsum(lens)])
        l = -rng.exponential(0.2, size=int(off[-1]))
        s = span_confidence(l, off)
        for p in range(n):
            want = 1.0
            for r in range(int(off[p]) + 1, int(off[p + 1])):
                want = min(want, math.exp(l[r]))
            assert s[p] == pytest.approx(want, rel=1e-14, abs=0)


def test_first_row_is_not_scored():
    # a span whose first row is very uncertain still commits on the rest
    l = np.log(np.array([0.05, 0.99, 0.93]))
    assert span_confidence(l, [0, 3])[0] == pytest.approx(0.93)
    assert confidence_gate(span_confidence(l, [0, 3]), 0.90).tolist() == [True]
    assert confidence_gate([0.8999999, 0.9, 0.95], 0.90).tolist() == [False, True, True]
