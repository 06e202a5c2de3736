"""Pins for the oracle greedy argmax and longest-prefix accept (Section 4.3).

References: numpy.argmax (documented to return the first occurrence of the
maximum), a hand-worked trace with ties and signed zeros, the synthetic
generator's planted greedy tokens and match counts (known by construction,
without computing an argmax), and a brute-force first-mismatch scan.
"""
import json
import os

import numpy as np
import pytest

from oracle import argmax_rows, accept_drafts
from paper_2607_03333_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_trace():
    with open(os.path.join(GOLDEN, "accept_trace.json")) as f:
        g = json.load(f)
    greedy = argmax_rows(np.array(g["logits"]))
    assert greedy.tolist() == g["expect_greedy"]
    a, n = accept_drafts(greedy, np.array(g["drafts"]))
    assert a.tolist() == g["expect_accept"] and n.tolist() == g["expect_next"]


def test_argmax_matches_numpy_first_occurrence():
    rng = np.random.default_rng(21)
    x = rng.integers(-3, 4, size=(200, 37)).astype(np.float64)  # many ties
    assert np.array_equal(argmax_rows(x), np.argmax(x, axis=1))
    y = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(rng.standard_normal((50, 4096)).astype(np.float32)))
    assert np.array_equal(argmax_rows(y), np.argmax(y, axis=1))


def test_argmax_brute_force_scan():
    rng = np.random.default_rng(22)
    x = rng.integers(0, 3, size=(40, 9)).astype(np.float32)
    x[rng.random(x.shape) < 0.2] *= -1.0
    for r in range(x.shape[0]):
        best, idx = -np.inf, -1
        for j in range(x.shape[1]):
            if x[r, j] > best:
                best, idx = x[r, j], j
        assert argmax_rows(x[r:r + 1])[0] == idx


def test_accept_brute_force():
    rng = np.random.default_rng(23)
    for _ in range(200):
        s, k = rng.integers(1, 5), rng.integers(1, 8)
        g = rng.integers(0, 3, size=s * (k + 1))
        d = rng.integers(0, 3, size=(s, k))
        a, n = accept_drafts(g, d)
        gg = g.reshape(s, k + 1)
        for i in range(s):
            m = 0
            while m < k and gg[i, m] == d[i, m]:
                m += 1
            assert a[i] == m and n[i] == gg[i, m]
            # committed tokens are the greedy tokens (lossless verification)
            committed = list(d[i, :a[i]]) + [n[i]]
            assert committed == list(gg[i, : a[i] + 1])


def test_all_match_and_none_match():
    g = np.array([5, 6, 7, 8, 1, 2, 3, 4])
    a, n = accept_drafts(g, np.array([[5, 6, 7], [9, 2, 3]]))
    assert a.tolist() == [3, 0] and n.tolist() == [8, 1]


@pytest.mark.parametrize("index,shrink", [
    (0, {}),
    (3, dict(sessions=6, prefix=32, vocab=3000)),
    (4, dict(sessions=8, prefix=32, suffix=("uniform", 1, 20), vocab=4096)),
])
def test_planted_ground_truth(index, shrink):
    wl = synth.make(index, **shrink)
    step = wl.steps[-1]
    g = argmax_rows(synth.to_f64(step.logits, wl.logits_dtype))
    assert np.array_equal(g, step.planted_greedy)
    a, n = accept_drafts(g, step.drafts)
    assert np.array_equal(a, step.planted_accept)
    assert np.array_equal(n, step.planted_next)
    if index == 0:
        assert a.tolist() == [2]
