"""Oracle attention: exact softmax attention of main, probe and verify rows.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What is computed (the plain definition; forking and cascading only change
where the bytes come from, Section 4.1):

For a thread with context ``K, V`` of ``L`` tokens (``[L, Hkv, D]``) and ``n``
query rows ``q`` (``[n, Hq, D]``), row ``r`` sits at position ``L - n + r``:
decode threads have ``n = 1`` (the newest token); a verify thread has
``n = K + 1`` rows, the last committed token followed by the ``K`` draft tokens
that the engine checks in one step (Section 4.3, step 2). Row ``r`` attends to
context positions ``0 .. L - n + r`` (bottom-right causal rule). Query head
``h`` reads KV head ``h // (Hq / Hkv)`` (grouped-query attention; the paper
names no head layout, contiguous groups is this project's reading).

    s_j  = scale * <q[r, h], K[j, h // G]>          j = 0 .. L - n + r
    m    = max_j s_j
    l    = sum_j exp(s_j - m)
    o    = sum_j exp(s_j - m) * V[j, h // G] / l
    lse  = m + ln l

Everything in float64; bf16 inputs are upcast exactly before use.

Parity pins (tests/test_oracle_attention.py): torch's CPU
``scaled_dot_product_attention`` in float64 with an explicit mask; closed forms
(constant V, identical keys, one dominant key, a single token, zero query);
a hand-worked two-token example under ``tests/golden/``; softmax weights sum to
one; splitting the context and merging by log-sum-exp; GQA head mapping with
per-head constant V; verify row ``r`` equals a decode on the context cut at its
position.
"""

import numpy as np


def attend(q, k, v, scale, return_weights=False):
    """Attention of ``n`` rows over one thread's contiguous context.

    ``q``: ``[n, Hq, D]``; ``k``, ``v``: ``[L, Hkv, D]``; all cast to float64.
    Returns ``o`` ``[n, Hq, D]`` and ``lse`` ``[n, Hq]`` (natural log), and the
    weights ``[n, Hq, L]`` (zero past each row's position) when asked.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    n, hq, d = q.shape
    length, hkv, _ = k.shape
    if hq % hkv != 0:
        raise ValueError("Hq must be a multiple of Hkv")
    if n > length:
        raise ValueError("a thread cannot have more query rows than context tokens")
    group = hq // hkv
    o = np.zeros((n, hq, d))
    lse = np.zeros((n, hq))
    weights = np.zeros((n, hq, length)) if return_weights else None
    for r in range(n):
        last = length - n + r           # inclusive horizon of row r
        for h in range(hq):
            kh = k[: last + 1, h // group, :]
            vh = v[: last + 1, h // group, :]
            s = scale * (kh @ q[r, h])
            m = s.max()
            p = np.exp(s - m)
            l = p.sum()
            o[r, h] = (p @ vh) / l
            lse[r, h] = m + np.log(l)
            if return_weights:
                weights[r, h, : last + 1] = p / l
    if return_weights:
        return o, lse, weights
    return o, lse


def attend_batch(q, contexts, n_rows, scale):
    """Attention for a batch of threads whose rows are stacked in ``q``.

    ``contexts[t] = (K_t, V_t)``; thread ``t`` owns the next ``n_rows[t]`` rows
    of ``q`` in order. Returns stacked ``o`` and ``lse``.
    """
    outs, lses = [], []
    row = 0
    for (k, v), n in zip(contexts, n_rows):
        o, lse = attend(q[row:row + n], k, v, scale)
        outs.append(o)
        lses.append(lse)
        row += n
    if row != q.shape[0]:
        raise ValueError("n_rows does not cover q")
    return np.concatenate(outs), np.concatenate(lses)
