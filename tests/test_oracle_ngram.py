"""Pins for the oracle n-gram (prompt-lookup) draft proposer.

References: a hand-worked trace, a second implementation over numpy sliding
windows, closed forms for periodic sequences and for sequences without a
repeat.
"""
import json
import os

import numpy as np
import pytest
from numpy.lib.stride_tricks import sliding_window_view

from oracle import ngram_propose, ngram_propose_one

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_trace():
    with open(os.path.join(GOLDEN, "ngram_trace.json")) as f:
        g = json.load(f)
    for c in g["cases"]:
        d, n = ngram_propose_one(c["tokens"], g["n_min"], g["n_max"], g["k"])
        assert d.tolist() == c["drafts"] and n == c["n"], c["why"]


def _windows(t, n_min, n_max, k):
    """The same lookup with whole-array window comparisons."""
    t = np.asarray(t, dtype=np.int64)
    L = len(t)
    for n in range(n_max, n_min - 1, -1):
        if L - 1 < n:
            continue
        w = sliding_window_view(t[: L - 1], n)          # windows with a token after them
        hit = np.nonzero((w == t[L - n:]).all(axis=1))[0]
        if hit.size:
            j = int(hit.max())
            f = t[j + n: j + n + k]
            return np.concatenate([f, np.full(k - f.size, -1)]), int(f.size)
    return np.full(k, -1), 0


@pytest.mark.parametrize("alphabet,n_min,n_max,k", [(2, 1, 3, 5), (3, 2, 4, 8), (5, 1, 1, 3), (4, 3, 5, 1)])
def test_matches_sliding_windows(alphabet, n_min, n_max, k):
    rng = np.random.default_rng(alphabet * 100 + n_max)
    for _ in range(300):
        t = rng.integers(0, alphabet, size=int(rng.integers(0, 40)))
        d, n = ngram_propose_one(t, n_min, n_max, k)
        wd, wn = _windows(t, n_min, n_max, k)
        assert n == wn and np.array_equal(d, wd), t.tolist()


@pytest.mark.parametrize("q", [1, 2, 5, 13])
def test_periodic_sequence_continues_its_period(q):
    # tokens i mod q: the latest occurrence of the key ends q positions back,
    # so the drafts are the next k tokens of the period (cut at the end)
    n_max, k = 4, 7
    L = 3 * q + n_max + 2
    t = np.arange(L) % q
    d, n = ngram_propose_one(t, 1, n_max, k)
    m = min(k, q)                                    # tokens after an occurrence ending q back
    assert n == m
    assert d[:m].tolist() == [(L + i) % q for i in range(m)]


def test_no_repeat_no_drafts():
    d, n = ngram_propose_one(np.arange(1000), 1, 5, 8)
    assert n == 0 and d.tolist() == [-1] * 8


def test_batch_form_and_key_never_matches_itself():
    seqs = [[1, 2, 3], [4, 4], [], [8, 9, 8, 9]]
    d, n = ngram_propose(seqs, 1, 2, 3)
    assert n.tolist() == [0, 1, 0, 2]
    assert d[1].tolist() == [4, -1, -1] and d[3].tolist() == [8, 9, -1]
