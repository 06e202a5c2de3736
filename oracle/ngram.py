"""Oracle n-gram (prompt-lookup) draft proposer.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper basis: the baseline the paper builds on is the serving engine's
model-free n-gram speculative decoding, which drafts from n-grams of the
prompt and of the output so far (Section 6.1 "Configurations"; Section 7,
token-level speculative decoding); D3's proposer wraps that same proposer and
substitutes the probe's tool call at the tool-call opener (Section 4.3).

The paper does not spell out the lookup; the readings used here:

* the lookup key is the last ``n`` tokens of the sequence, for ``n`` from
  ``n_max`` down to ``n_min``; the first ``n`` with an earlier occurrence wins;
* an occurrence is a start ``j`` with ``tokens[j:j+n] == tokens[L-n:L]`` and at
  least one token after it (``j + n <= L - 1``), so the key itself never
  matches; occurrences may overlap the key;
* among occurrences the latest (largest ``j``) wins;
* the drafts are the up to ``k`` tokens that follow the occurrence, cut at the
  end of the sequence; missing drafts are padded with -1, a value no greedy
  token takes, so the verify step accepts at most the real drafts.

Parity pins: a vectorised search over ``numpy`` sliding windows (a second
implementation), closed forms for periodic sequences, sequences without
repeats, the cut at the end, and a hand-worked trace in
``tests/golden/ngram_trace.json``.
"""

import numpy as np


def ngram_propose_one(tokens, n_min, n_max, k):
    """Drafts (length k, -1 padded) and their count for one token sequence."""
    t = [int(x) for x in tokens]
    L = len(t)
    out = [-1] * k
    for n in range(n_max, n_min - 1, -1):
        if n > L - 1:
            continue
        key = t[L - n:]
        for j in range(L - n - 1, -1, -1):
            if t[j:j + n] == key:
                follow = t[j + n: j + n + k]
                out[:len(follow)] = follow
                return np.array(out, dtype=np.int64), len(follow)
    return np.array(out, dtype=np.int64), 0


def ngram_propose(seqs, n_min, n_max, k):
    """Batch form: ``seqs`` is a list of token sequences; returns drafts
    ``[S, k]`` and counts ``[S]``."""
    drafts = np.full((len(seqs), k), -1, dtype=np.int64)
    counts = np.zeros(len(seqs), dtype=np.int64)
    for i, s in enumerate(seqs):
        drafts[i], counts[i] = ngram_propose_one(s, n_min, n_max, k)
    return drafts, counts
