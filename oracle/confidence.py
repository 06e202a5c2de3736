"""Oracle top-1 log-probability and the D2 confidence gate.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper basis: Section 4.2 (D2, the adaptive confidence gate). The probe
generates its tool-call tokens with per-token log-probabilities; the confidence
score is the smallest top-1 token probability exp(l_i) over the tool-name span
without its first token (the opening quote, always likely), l_i being the
log-probability of the top-1 token at span position i; the probe commits to a
speculative tool dispatch once the score reaches the threshold theta (the
paper settles on 0.90). Decoding is greedy (Section 6.1), so the top-1 token is
the greedy token.

Readings used here:

* ``l = x_max - log(sum_v exp(x_v))`` over a position's logits ``x`` (the
  log-softmax of the greedy token), computed in float64;
* a probe's span is a run of consecutive rows ``[off[p], off[p + 1])``; its
  score is ``min(exp(l[r]))`` over rows ``off[p] + 1 .. off[p + 1] - 1``; a span
  of fewer than two tokens leaves an empty set, whose score is taken as 1 (the
  identity of the minimum over probabilities);
* the gate commits when ``score >= theta``.

Parity pins: ``scipy.special.logsumexp`` (an independent implementation);
closed forms (equal logits give ``-log V``; two tied maxima far above the rest
give ``-log 2``; a maximum ``d`` above ``V - 1`` equal others gives
``-log(1 + (V - 1) e^-d)``); the softmax probability of the argmax token from
``torch.softmax`` in float64; a hand-worked span trace in
``tests/golden/confidence_trace.json``.
"""

import numpy as np


def top1_logprob(logits):
    """Log-probability of each row's top-1 token (``logits`` 2-D, any real dtype)."""
    x = np.asarray(logits, dtype=np.float64)
    m = x.max(axis=1, keepdims=True)
    return -np.log(np.exp(x - m).sum(axis=1))


def span_confidence(logprob, span_off):
    """Smallest top-1 probability over each span without its first row (1 if empty)."""
    l = np.asarray(logprob, dtype=np.float64)
    off = np.asarray(span_off, dtype=np.int64)
    out = np.ones(len(off) - 1, dtype=np.float64)
    for p in range(len(off) - 1):
        rows = range(off[p] + 1, off[p + 1])
        if len(rows):
            out[p] = min(np.exp(l[r]) for r in rows)
    return out


def confidence_gate(score, theta):
    """Commit decision of each probe."""
    return np.asarray(score, dtype=np.float64) >= theta
