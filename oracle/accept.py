"""Oracle greedy argmax and longest-prefix draft accept.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper basis: decoding is greedy (temperature 0; Section 6.1 "Setup"). In D3
(Section 4.3, steps 2-3) the rejected probe's tool-call body is the draft; the
engine verifies it in one decode step, accepts the longest draft prefix that
equals the main model's greedy tokens, and resumes after the first mismatch
(Appendix B reports the first-mismatch position k on real traces).

Reading used here, for ``S`` verify threads with ``K`` drafts each and logits
``[S * (K + 1), V]`` (row ``s * (K + 1) + r`` is verify row ``r`` of thread ``s``):

* ``g[row]`` = the lowest vocabulary index holding the row maximum (the paper is
  silent on ties; lowest index is the first-occurrence rule of numpy/torch);
  values compare after exact upcast, so +0 and -0 tie;
* ``a_s`` = the first ``r < K`` with ``g[s, r] != d[s, r]``, else ``K``;
* ``next_s`` = ``g[s, a_s]`` (the corrected token, or the bonus token when every
  draft matched); the committed tokens are ``d[s, :a_s]`` then ``next_s``,
  which equal ``g[s, :a_s + 1]`` (verification is lossless, Section 6.3).

Parity pins: ``numpy.argmax`` (documented first-occurrence semantics) and a
pure-Python scan on planted ties; the synthetic generator's planted match counts
(known by construction); the first-mismatch brute force.
"""

import numpy as np


def argmax_rows(logits):
    """Lowest index attaining each row's maximum (``logits`` 2-D, any real dtype)."""
    x = np.asarray(logits, dtype=np.float64)
    best = x.max(axis=1, keepdims=True)
    hit = x == best
    return hit.argmax(axis=1).astype(np.int64)


def accept_drafts(g, drafts):
    """Accepted length and next token per verify thread.

    ``g``: ``[S * (K + 1)]`` greedy tokens; ``drafts``: ``[S, K]``.
    """
    drafts = np.asarray(drafts)
    s_count, k = drafts.shape
    g = np.asarray(g).reshape(s_count, k + 1)
    accept = np.empty(s_count, dtype=np.int64)
    nxt = np.empty(s_count, dtype=np.int64)
    for s in range(s_count):
        a = k
        for r in range(k):
            if g[s, r] != drafts[s, r]:
                a = r
                break
        accept[s] = a
        nxt[s] = g[s, a]
    return accept, nxt
