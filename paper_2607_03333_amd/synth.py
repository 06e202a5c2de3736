"""Seeded synthetic workloads for the forked-decode hot path.

This module only draws numbers and lays out a scenario; it holds none of the
method's arithmetic (no attention, no argmax, no accept, no block allocation).
The product path, the tests and the oracle all take their inputs from here.

The paper measures on agent benchmarks with Qwen3 models served by vLLM
(Section 6.1); neither the benchmarks nor the weights are available, so seeded
Gaussian data with the workload's structure stands in for them:

* one shared prefix per session (the system + user + history prompt that D1's
  fork reuses, Section 4.1; about 15K tokens of context in the paper's
  measurement of probe cost);
* a main thread plus forked probes per session, each with a private suffix
  (the chain of thought between the fork and the tool call is about 2,000
  tokens, Section 1);
* verify threads that carry ``K`` draft rows (the rejected probe's tool-call
  body, Section 4.3) and greedy logits whose argmax is planted by construction:
  every row has a value above all others at a chosen index, sometimes at two
  indices (a tie), so the greedy token and the expected accepted length are
  known without computing an argmax.

Seeds (42 is the seed the paper uses for every call, Section 6.1): the
workload stream ``numpy.random.default_rng([42, index])`` draws, in order, the
suffix lengths, the pool free order, per-step Q, then per verify step the
planted greedy tokens and ties, match counts and drafts. Bulk arrays come from
their own streams so they can be drawn in parallel: session ``s``'s prefix K
then V from ``[42, index, 1, s]``, sequence ``t``'s private K then V from
``[42, index, 2, t]``, verify step ``j``'s raw logits from ``[42, index, 3, j]``.
"""

import os
from concurrent.futures import ThreadPoolExecutor

from dataclasses import dataclass, field
import math

import numpy as np

F32 = "f32"
BF16 = "bf16"

# The five workloads of the benchmark, by what they are (sizes stated in full).
CONFIGS = [
    dict(name="tiny-fork-f32", hq=4, hkv=2, d=64, block_size=16, dtype=F32,
         sessions=1, probes=1, prefix=256, suffix=("fixed", [32, 8]),
         verify_k=4, vocab=512, logits_dtype=F32, planted_n="fixed2",
         q_scale_in_softmax=0.125, layout="decode-then-verify"),
    dict(name="qwen3-4b-decode", hq=32, hkv=8, d=128, block_size=16, dtype=BF16,
         sessions=8, probes=1, prefix=4096, suffix=("uniform", 1, 2048),
         verify_k=0, vocab=0, logits_dtype=BF16, layout="decode"),
    dict(name="qwen3-32b-decode", hq=64, hkv=8, d=128, block_size=16, dtype=BF16,
         sessions=16, probes=4, prefix=16384, suffix=("uniform", 1, 2000),
         verify_k=0, vocab=0, logits_dtype=BF16, layout="decode"),
    dict(name="qwen3-32b-verify", hq=64, hkv=8, d=128, block_size=16, dtype=BF16,
         sessions=16, probes=0, prefix=16384, suffix=("fixed", [0]),
         verify_k=16, vocab=151936, logits_dtype=BF16, planted_n="geom0.3",
         layout="verify"),
    dict(name="qwen3-30b-a3b-mixed", hq=32, hkv=4, d=128, block_size=16, dtype=BF16,
         sessions=64, probes=2, prefix=32768, suffix=("loguniform", 1, 4096),
         verify_k=8, vocab=151936, logits_dtype=BF16, planted_n="geom0.3",
         layout="mixed"),
]

PLANT_VALUE = 7.0     # planted greedy logit; every other logit is clipped to [-6, 6]
CLIP = 6.0
TIE_PROB = 0.25       # chance that a row carries a second planted maximum


def config_index(name_or_index):
    if isinstance(name_or_index, int):
        return name_or_index
    for i, c in enumerate(CONFIGS):
        if c["name"] == name_or_index:
            return i
    raise KeyError(name_or_index)


# --- storage conversions (exact bit operations, no rounding choices beyond RNE) ---
def f32_to_bf16_bits(x):
    """Round float32 to bfloat16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_storage(x, dtype):
    return f32_to_bf16_bits(x) if dtype == BF16 else np.ascontiguousarray(x, dtype=np.float32)


def to_f64(x, dtype):
    """Exact upcast of stored values to float64."""
    if dtype == BF16:
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float64)


@dataclass
class Thread:
    seq: int            # sequence id (ids are issued 0, 1, 2, ... in creation order)
    session: int
    role: str           # "main" or "probe"
    suffix: int         # private tokens appended after the fork (includes the decode token)
    drafts: int = 0     # draft tokens appended before the verify step
    parent: int = -1    # sequence forked from (-1: a root that owns its session prefix)
    fork_len: int = 0   # parent's context length at the fork


@dataclass
class Step:
    """One call of the hot path: the threads, their rows and groups, Q, and verify data."""
    seqs: list
    n_rows: list
    groups: list
    q: np.ndarray                       # [rows, Hq, D] in storage dtype
    ops_before: list                    # scenario ops to apply before this step
    logits: np.ndarray = None           # [S*(K+1), V] storage dtype
    drafts: np.ndarray = None           # [S, K] int32
    planted_greedy: np.ndarray = None   # [S*(K+1)] greedy token per row, by construction
    planted_accept: np.ndarray = None   # [S]
    planted_next: np.ndarray = None     # [S]
    verify_k: int = 0


def draw_kv(seed, n, hkv, d, dtype):
    """K then V of ``n`` tokens from the stream ``default_rng(seed)``, storage dtype."""
    r = np.random.default_rng(seed)
    k = to_storage(r.standard_normal((n, hkv, d), dtype=np.float32), dtype)
    v = to_storage(r.standard_normal((n, hkv, d), dtype=np.float32), dtype)
    return k, v


def _draw_segments(segs, hkv, d, dtype):
    pairs = [draw_kv(seed, n, hkv, d, dtype) for seed, n in segs]
    if len(pairs) == 1:
        return pairs[0]
    return np.concatenate([p[0] for p in pairs]), np.concatenate([p[1] for p in pairs])


@dataclass
class Workload:
    index: int
    name: str
    hq: int
    hkv: int
    d: int
    block_size: int
    dtype: str
    logits_dtype: str
    sm_scale: float
    num_blocks: int
    free_order: np.ndarray
    threads: list
    prefix_len: list                    # per session
    prefix_k: list                      # per session [P, Hkv, D] storage dtype
    prefix_v: list
    suffix_k: dict                      # per seq [suffix + drafts, Hkv, D]
    suffix_v: dict
    steps: list = field(default_factory=list)
    # Where every K/V array comes from: ("p", session) and ("s", seq) map to
    # segments (seed, tokens), each drawn K then V from default_rng(seed).
    # Without stored arrays (built with kv=False) they are drawn on demand.
    kv_src: dict = field(default_factory=dict)
    _kv_cache: dict = field(default_factory=dict, repr=False)

    def thread(self, seq):
        return next(t for t in self.threads if t.seq == seq)

    def _lazy(self, key):
        if key not in self._kv_cache:
            if len(self._kv_cache) >= 8:
                self._kv_cache.pop(next(iter(self._kv_cache)))
            self._kv_cache[key] = _draw_segments(self.kv_src[key], self.hkv, self.d, self.dtype)
        return self._kv_cache[key]

    def prefix_kv(self, session):
        if self.prefix_k is not None:
            return self.prefix_k[session], self.prefix_v[session]
        return self._lazy(("p", session))

    def suffix_kv(self, seq):
        if self.suffix_k is not None:
            return self.suffix_k[seq], self.suffix_v[seq]
        return self._lazy(("s", seq))

    def context(self, seq, length=None):
        """Logical K, V of a thread, storage dtype: a root's session prefix, or
        its parent's context up to the fork, then its own tokens."""
        t = self.thread(seq)
        if t.parent >= 0:
            pk, pv = self.context(t.parent, t.fork_len)
        else:
            pk, pv = self.prefix_kv(t.session)
        sk, sv = self.suffix_kv(seq)
        k = np.concatenate([pk, sk])
        v = np.concatenate([pv, sv])
        if length is not None:
            k, v = k[:length], v[:length]
        return k, v

    def thread_len(self, seq, upto_step):
        """Context length of ``seq`` when step ``upto_step`` runs."""
        n = 0
        for step in self.steps[: upto_step + 1]:
            for op in step.ops_before:
                if op[0] == "append" and op[1] == seq:
                    n += op[2]
                if op[0] == "fork" and op[2] == seq:
                    n += self._len_at_fork(op[1], step, op)
        return n

    def _len_at_fork(self, parent, step, fork_op):
        n = 0
        for st in self.steps:
            for op in st.ops_before:
                if op is fork_op:
                    return n
                if op[0] == "append" and op[1] == parent:
                    n += op[2]
        return n

    def unique_kv_bytes(self, step_index):
        """KV bytes a step must read once: every stored token that one of the
        step's threads sees, once. A forked thread shares its parent's blocks
        up to the block holding the fork point; from that block on its tokens
        are its own copy (the block is copied on the first write)."""
        step = self.steps[step_index]
        elem = 4 if self.dtype == F32 else 2
        per_tok = 2 * self.hkv * self.d * elem
        bs = self.block_size

        def own_lo(t):
            return 0 if t.parent < 0 else (t.fork_len // bs) * bs

        upper = {}
        for s in step.seqs:
            t, hi = self.thread(s), self.thread_len(s, step_index)
            while True:
                upper[t.seq] = max(upper.get(t.seq, 0), hi)
                if t.parent < 0:
                    break
                hi, t = own_lo(t), self.thread(t.parent)
        total = sum(max(0, hi - own_lo(self.thread(q))) for q, hi in upper.items())
        return total * per_tok


def _draw_all(kv_src, prefix_keys, seqs, hkv, d, dtype, kv):
    """Stored K/V arrays of a workload (prefixes by session, suffixes by
    sequence), drawn in parallel; all None when ``kv`` is false."""
    if not kv:
        return None, None, None, None
    keys = list(prefix_keys) + [("s", q) for q in seqs]
    with ThreadPoolExecutor(max(1, min(16, os.cpu_count() or 1))) as ex:
        pairs = list(ex.map(lambda key: _draw_segments(kv_src[key], hkv, d, dtype), keys))
    n_p = len(prefix_keys)
    return ([p[0] for p in pairs[:n_p]], [p[1] for p in pairs[:n_p]],
            {q: pairs[n_p + i][0] for i, q in enumerate(seqs)}, {q: pairs[n_p + i][1] for i, q in enumerate(seqs)})


def _draw_suffix(rng, spec, n):
    kind = spec[0]
    if kind == "fixed":
        vals = list(spec[1])
        return [vals[i % len(vals)] for i in range(n)]
    if kind == "uniform":
        return [int(x) for x in rng.integers(spec[1], spec[2] + 1, size=n)]
    if kind == "loguniform":
        lo, hi = spec[1], spec[2]
        u = rng.uniform(0.0, math.log(hi + 1), size=n)
        return [int(min(max(math.floor(math.exp(x)), lo), hi)) for x in u]
    raise ValueError(kind)


def make(index, sessions=None, prefix=None, suffix=None, vocab=None, verify_k=None,
         block_size=None, q_gain=1.0, tie_prob=TIE_PROB, kv=True):
    """Build workload ``index`` (0..4), optionally shrunk for fast tests.

    Overrides keep the workload's structure (forks, rows, GQA, dtype) while
    changing its size. ``q_gain`` multiplies Q (a sharper softmax). With
    ``kv=False`` no K/V array is drawn up front; ``context`` draws a
    thread's from its own seed streams when asked (same values).
    """
    index = config_index(index)
    cfg = dict(CONFIGS[index])
    if sessions is not None:
        cfg["sessions"] = sessions
    if prefix is not None:
        cfg["prefix"] = prefix
    if suffix is not None:
        cfg["suffix"] = suffix
    if vocab is not None:
        cfg["vocab"] = vocab
    if verify_k is not None:
        cfg["verify_k"] = verify_k
    if block_size is not None:
        cfg["block_size"] = block_size
    rng = np.random.default_rng([42, index])
    hq, hkv, d, bs, dtype = cfg["hq"], cfg["hkv"], cfg["d"], cfg["block_size"], cfg["dtype"]
    n_sess, n_probe, plen = cfg["sessions"], cfg["probes"], cfg["prefix"]
    kd = cfg["verify_k"]
    layout = cfg["layout"]
    if "q_scale_in_softmax" in cfg:
        sm_scale = float(np.float32(cfg["q_scale_in_softmax"]))
    else:
        sm_scale = float(np.float32(1.0 / math.sqrt(d)))

    # Threads: mains get ids 0..S-1, probes follow in session order.
    threads = []
    for s in range(n_sess):
        threads.append(Thread(seq=s, session=s, role="main", suffix=0))
    nid = n_sess
    for s in range(n_sess):
        for _ in range(n_probe):
            threads.append(Thread(seq=nid, session=s, role="probe", suffix=0, parent=s, fork_len=plen))
            nid += 1
    by_session = {s: [t for t in threads if t.session == s] for s in range(n_sess)}
    ordered = [t for s in range(n_sess) for t in by_session[s]]   # main, probes per session
    lens = _draw_suffix(rng, cfg["suffix"], len(ordered))
    for t, n in zip(ordered, lens):
        t.suffix = n
    verify_threads = []
    if layout in ("verify", "mixed", "decode-then-verify"):
        for s in range(n_sess):
            by_session[s][0].drafts = kd
            verify_threads.append(by_session[s][0])

    blocks = sum(-(-plen // bs) for _ in range(n_sess))
    blocks += sum(-(-(t.suffix + t.drafts) // bs) + 1 for t in threads)
    num_blocks = blocks + 16
    free_order = rng.permutation(num_blocks).astype(np.int32)

    def normal(shape, r=rng):
        return r.standard_normal(shape, dtype=np.float32)

    kv_src = {("p", s_): [([42, index, 1, s_], plen)] for s_ in range(n_sess)}
    kv_src.update({("s", t.seq): [([42, index, 2, t.seq], t.suffix + t.drafts)] for t in ordered})
    prefix_k, prefix_v, suffix_k, suffix_v = _draw_all(kv_src, [("p", s_) for s_ in range(n_sess)],
                                                       [t.seq for t in ordered], hkv, d, dtype, kv)

    build_ops = [("new", t.seq) for t in threads if t.role == "main"]
    build_ops += [("append", t.seq, plen) for t in threads if t.role == "main"]
    build_ops += [("fork", by_session[t.session][0].seq, t.seq) for t in threads if t.role == "probe"]
    build_ops += [("append", t.seq, t.suffix) for t in ordered if t.suffix > 0]
    draft_ops = [("append", t.seq, t.drafts) for t in verify_threads if t.drafts > 0]

    wl = Workload(index=index, name=cfg["name"], hq=hq, hkv=hkv, d=d, block_size=bs,
                  dtype=dtype, logits_dtype=cfg["logits_dtype"], sm_scale=sm_scale,
                  num_blocks=num_blocks, free_order=free_order, threads=threads,
                  prefix_len=[plen] * n_sess, prefix_k=prefix_k, prefix_v=prefix_v,
                  suffix_k=suffix_k, suffix_v=suffix_v, kv_src=kv_src)

    def q_for(n_rows_total):
        return to_storage(normal((n_rows_total, hq, d)) * np.float32(q_gain), dtype)

    def decode_step(ops):
        seqs = [t.seq for t in ordered]
        rows = [1] * len(seqs)
        groups = [t.session for t in ordered]
        return Step(seqs=seqs, n_rows=rows, groups=groups, q=q_for(len(seqs)), ops_before=ops)

    if layout == "decode":
        wl.steps.append(decode_step(build_ops))
    elif layout == "decode-then-verify":
        wl.steps.append(decode_step(build_ops))
        seqs = [t.seq for t in verify_threads]
        rows = [kd + 1] * len(seqs)
        wl.steps.append(Step(seqs=seqs, n_rows=rows, groups=[t.session for t in verify_threads],
                             q=q_for(sum(rows)), ops_before=draft_ops, verify_k=kd))
    elif layout == "verify":
        seqs = [t.seq for t in verify_threads]
        rows = [kd + 1] * len(seqs)
        wl.steps.append(Step(seqs=seqs, n_rows=rows, groups=[t.session for t in verify_threads],
                             q=q_for(sum(rows)), ops_before=build_ops + draft_ops, verify_k=kd))
    elif layout == "mixed":
        seqs = [t.seq for t in ordered]
        rows = [kd + 1 if t.drafts else 1 for t in ordered]
        wl.steps.append(Step(seqs=seqs, n_rows=rows, groups=[t.session for t in ordered],
                             q=q_for(sum(rows)), ops_before=build_ops + draft_ops, verify_k=kd))
    else:
        raise ValueError(layout)

    # Verify data: planted greedy tokens, ties, match counts and drafts.
    for j, step in enumerate(wl.steps):
        if step.verify_k == 0:
            continue
        vocab = cfg["vocab"]
        n_ver = len(verify_threads)
        rows = n_ver * (kd + 1)
        raw = np.clip(normal((rows, vocab), np.random.default_rng([42, index, 3, j])), -CLIP, CLIP)
        target = rng.integers(0, vocab, size=rows)
        tie = rng.random(rows) < tie_prob
        partner = (target + 1 + rng.integers(0, vocab - 1, size=rows)) % vocab
        raw[np.arange(rows), target] = PLANT_VALUE
        raw[np.arange(rows)[tie], partner[tie]] = PLANT_VALUE
        greedy = np.where(tie, np.minimum(target, partner), target).astype(np.int64)
        if cfg.get("planted_n") == "fixed2":
            n_match = np.full(n_ver, 2, dtype=np.int64)
        else:
            n_match = rng.geometric(0.3, size=n_ver).astype(np.int64) - 1
        n_match = np.minimum(n_match, kd)
        drafts = rng.integers(0, vocab, size=(n_ver, kd)).astype(np.int64)
        g = greedy.reshape(n_ver, kd + 1)
        for s in range(n_ver):
            drafts[s, : n_match[s]] = g[s, : n_match[s]]
            if n_match[s] < kd:
                drafts[s, n_match[s]] = (g[s, n_match[s]] + 1 + rng.integers(0, vocab - 1)) % vocab
        step.logits = to_storage(raw, cfg["logits_dtype"])
        step.drafts = drafts.astype(np.int32)
        step.planted_greedy = greedy
        step.planted_accept = n_match
        step.planted_next = g[np.arange(n_ver), n_match]
    return wl


@dataclass
class ProbeBatch:
    """Logits of probe positions grouped into tool-name spans."""
    logits: np.ndarray      # [n_rows, vocab] storage dtype
    span_off: np.ndarray    # [n_probes + 1] int32, span p = rows span_off[p] .. span_off[p+1]-1
    vocab: int
    dtype: str


def probe_batch(n_probes, vocab, dtype=BF16, span=(0, 12), seed=0, tie_prob=0.05, neg_inf_prob=0.0):
    """Probe positions of a D2 confidence check (Section 4.2).

    Span lengths are uniform in ``span`` (inclusive; 0 and 1 leave nothing to
    score). Each row is standard normal logits plus a boost on one random
    token of ln(vocab) + 0.5 + u, u uniform in [-4, 8], which spreads the
    top-1 probability from about 0.02 to above 0.999 (around 0.9 near
    u = 2.2); with probability ``tie_prob`` a second token gets the same boost
    (a tie), and each entry is -inf with probability ``neg_inf_prob`` (a
    masked vocabulary entry; the boosted tokens never are). Drawn from
    ``numpy.random.default_rng([42, 5, seed])``.
    """
    rng = np.random.default_rng([42, 5, seed])
    lens = rng.integers(span[0], span[1] + 1, size=n_probes)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    rows = int(off[-1])
    x = rng.standard_normal((rows, vocab)).astype(np.float32)
    if neg_inf_prob > 0:
        x[rng.random((rows, vocab)) < neg_inf_prob] = -np.inf
    boost = (math.log(vocab) + 0.5 + rng.uniform(-4.0, 8.0, size=rows)).astype(np.float32)
    target = rng.integers(0, vocab, size=rows)
    tie = rng.random(rows) < tie_prob
    partner = (target + 1 + rng.integers(0, max(vocab - 1, 1), size=rows)) % vocab
    x[np.arange(rows), target] = boost
    x[np.arange(rows)[tie], partner[tie]] = boost[tie]
    return ProbeBatch(logits=to_storage(x, dtype), span_off=off, vocab=vocab, dtype=dtype)


TREE_NAME = "qwen3-30b-a3b-staggered"


def make_tree(sessions=32, prefix=32768, probes=4, stride=200, probe_tokens=(8, 64), main_extra=(1, 200),
              hq=32, hkv=4, d=128, block_size=16, dtype=BF16, q_gain=1.0, kv=True):
    """Staggered probes (Algorithm 1's retry loop): a decode step over a
    prefix tree of forks.

    Per session the main thread holds the ``prefix``-token prompt; after its
    first CoT token it forks probe 0, and after every further ``stride`` CoT
    tokens the next probe (Algorithm 1 forks probe r once the main thread has
    decoded r * s more tokens; the paper does not give s, and 200 puts the
    fork points in the middle of 16-token blocks). The main thread then
    decodes ``main_extra`` (uniform, inclusive) more tokens and every probe
    holds ``probe_tokens`` (uniform) of its own: the forced tool-call opener
    and the tool call decoded so far. Probe r therefore shares
    ``prefix + 1 + r * stride`` tokens with the main thread and with every
    later probe. The step decodes one row for every thread, the threads of a
    session forming one fork group. Default shapes are the Qwen3-30B-A3B
    attention (32 query heads, 4 KV heads, head dim 128, bf16). Seeds:
    ``default_rng([42, 6])`` for lengths, order and Q; K and V of the prefix
    and of each thread's own tokens from ``[42, 6, 1, s]`` and ``[42, 6, 2, seq]``.
    """
    index = 6
    rng = np.random.default_rng([42, index])
    bs = block_size
    threads = [Thread(seq=s, session=s, role="main", suffix=0) for s in range(sessions)]
    nid = sessions
    for s in range(sessions):
        for r in range(probes):
            threads.append(Thread(seq=nid, session=s, role="probe", suffix=0, parent=s,
                                  fork_len=prefix + 1 + r * stride))
            nid += 1
    by_session = {s: [t for t in threads if t.session == s] for s in range(sessions)}
    ordered = [t for s in range(sessions) for t in by_session[s]]
    extra = rng.integers(main_extra[0], main_extra[1] + 1, size=sessions)
    for s in range(sessions):
        by_session[s][0].suffix = 1 + max(probes - 1, 0) * stride + int(extra[s])
    own = rng.integers(probe_tokens[0], probe_tokens[1] + 1, size=sessions * probes)
    for t, n in zip([t for t in ordered if t.role == "probe"], own):
        t.suffix = int(n)

    blocks = sessions * -(-prefix // bs) + sum(-(-t.suffix // bs) + 2 for t in threads)
    num_blocks = blocks + 16
    free_order = rng.permutation(num_blocks).astype(np.int32)

    def normal(shape, r=rng):
        return r.standard_normal(shape, dtype=np.float32)

    kv_src = {("p", s_): [([42, index, 1, s_], prefix)] for s_ in range(sessions)}
    kv_src.update({("s", t.seq): [([42, index, 2, t.seq], t.suffix)] for t in ordered})
    prefix_k, prefix_v, suffix_k, suffix_v = _draw_all(kv_src, [("p", s_) for s_ in range(sessions)],
                                                       [t.seq for t in ordered], hkv, d, dtype, kv)

    ops = []
    for s in range(sessions):
        main = by_session[s][0]
        ops += [("new", main.seq), ("append", main.seq, prefix)]
    for s in range(sessions):
        main = by_session[s][0]
        done = 0
        for t in by_session[s][1:]:
            step = t.fork_len - prefix - done
            ops.append(("append", main.seq, step))
            done += step
            ops.append(("fork", main.seq, t.seq))
        ops.append(("append", main.seq, main.suffix - done))
    for t in ordered:
        if t.role == "probe":
            ops.append(("append", t.seq, t.suffix))

    wl = Workload(index=index, name=TREE_NAME, hq=hq, hkv=hkv, d=d, block_size=bs, dtype=dtype,
                  logits_dtype=dtype, sm_scale=float(np.float32(1.0 / math.sqrt(d))),
                  num_blocks=num_blocks, free_order=free_order, threads=threads,
                  prefix_len=[prefix] * sessions, prefix_k=prefix_k, prefix_v=prefix_v,
                  suffix_k=suffix_k, suffix_v=suffix_v, kv_src=kv_src)
    q = to_storage(normal((len(ordered), hq, d)) * np.float32(q_gain), dtype)
    wl.steps.append(Step(seqs=[t.seq for t in ordered], n_rows=[1] * len(ordered),
                         groups=[t.session for t in ordered], q=q, ops_before=ops))
    return wl


PREFILL_NAME = "qwen3-30b-a3b-probe-prefill"


def make_prefill(sessions=64, prefix=32768, probes=2, cot=("loguniform", 1, 4096), opener=(8, 50),
                 hq=32, hkv=4, d=128, block_size=16, dtype=BF16, q_gain=1.0, kv=True):
    """Probe prefill over the shared prefix (Section 4.1: the probe's prefill
    is a prefix-cache hit): one step in which every main thread decodes one
    row while its probes, just forked after the chain of thought observed so
    far, prefill their forced tool-call openers as multi-row causal queries.

    Per session the main thread holds a ``prefix``-token prompt and ``cot``
    tokens of chain of thought (log-uniform, as the bench workload's private
    suffixes); ``probes`` probes fork there; each probe then appends its
    opener of ``opener`` tokens (uniform, inclusive) and queries all of them,
    causally among themselves, while the main thread appends and queries its
    next token. Default shapes are the Qwen3-30B-A3B attention. Seeds:
    ``default_rng([42, 7])`` for lengths, order and Q; K and V from
    ``[42, 7, 1, session]`` and ``[42, 7, 2, seq]``.
    """
    index = 7
    rng = np.random.default_rng([42, index])
    bs = block_size
    cot_len = _draw_suffix(rng, cot, sessions)
    threads = [Thread(seq=s, session=s, role="main", suffix=cot_len[s] + 1) for s in range(sessions)]
    nid = sessions
    for s in range(sessions):
        for _ in range(probes):
            threads.append(Thread(seq=nid, session=s, role="probe", suffix=0, parent=s,
                                  fork_len=prefix + cot_len[s]))
            nid += 1
    by_session = {s: [t for t in threads if t.session == s] for s in range(sessions)}
    ordered = [t for s in range(sessions) for t in by_session[s]]
    op_len = rng.integers(opener[0], opener[1] + 1, size=sessions * probes)
    for t, n in zip([t for t in ordered if t.role == "probe"], op_len):
        t.suffix = int(n)

    blocks = sessions * -(-prefix // bs) + sum(-(-t.suffix // bs) + 2 for t in threads)
    num_blocks = blocks + 16
    free_order = rng.permutation(num_blocks).astype(np.int32)

    def normal(shape, r=rng):
        return r.standard_normal(shape, dtype=np.float32)

    kv_src = {("p", s_): [([42, index, 1, s_], prefix)] for s_ in range(sessions)}
    kv_src.update({("s", t.seq): [([42, index, 2, t.seq], t.suffix)] for t in ordered})
    prefix_k, prefix_v, suffix_k, suffix_v = _draw_all(kv_src, [("p", s_) for s_ in range(sessions)],
                                                       [t.seq for t in ordered], hkv, d, dtype, kv)

    ops = []
    for s in range(sessions):
        ops += [("new", s), ("append", s, prefix + cot_len[s])]
    for t in ordered:
        if t.role == "probe":
            ops.append(("fork", t.parent, t.seq))
    for t in ordered:
        ops.append(("append", t.seq, 1 if t.role == "main" else t.suffix))

    wl = Workload(index=index, name=PREFILL_NAME, hq=hq, hkv=hkv, d=d, block_size=bs, dtype=dtype,
                  logits_dtype=dtype, sm_scale=float(np.float32(1.0 / math.sqrt(d))),
                  num_blocks=num_blocks, free_order=free_order, threads=threads,
                  prefix_len=[prefix] * sessions, prefix_k=prefix_k, prefix_v=prefix_v,
                  suffix_k=suffix_k, suffix_v=suffix_v, kv_src=kv_src)
    rows = [1 if t.role == "main" else t.suffix for t in ordered]
    q = to_storage(normal((sum(rows), hq, d)) * np.float32(q_gain), dtype)
    wl.steps.append(Step(seqs=[t.seq for t in ordered], n_rows=rows, groups=[t.session for t in ordered],
                         q=q, ops_before=ops))
    return wl


def make_named(name, **kw):
    """Any workload by name: the five benchmark workloads, the staggered fork
    tree and the probe prefill."""
    if name == TREE_NAME:
        return make_tree(**kw)
    if name == PREFILL_NAME:
        return make_prefill(**kw)
    return make(name, **kw)


def token_histories(n_seqs, lengths, vocab=151936, seed=0, copy_prob=0.35, mean_segment=16):
    """Token sequences (prompt and output so far) for the n-gram draft
    proposer: concatenated segments of geometric length (mean
    ``mean_segment``), each with probability ``copy_prob`` a copy of an
    earlier span of the same sequence (agent traces repeat tool output, JSON
    keys and earlier calls), else fresh tokens of Zipf(1.2) rank (frequent
    tokens recur). ``lengths`` is a list or a (lo, hi) range drawn uniformly.
    Returns the concatenated int32 tokens and int64 offsets ``[n_seqs + 1]``.
    Drawn from ``numpy.random.default_rng([42, 8, seed])``."""
    rng = np.random.default_rng([42, 8, seed])
    if isinstance(lengths, tuple):
        lengths = rng.integers(lengths[0], lengths[1] + 1, size=n_seqs)
    seqs = []
    for L in lengths:
        L = int(L)
        t = np.empty(L, dtype=np.int32)
        n = 0
        while n < L:
            seg = min(int(rng.geometric(1.0 / mean_segment)), L - n)
            if n >= 2 and rng.random() < copy_prob:
                src = int(rng.integers(0, n - 1))
                seg = min(seg, n - src)
                t[n:n + seg] = t[src:src + seg]
            else:
                t[n:n + seg] = (rng.zipf(1.2, size=seg) - 1) % vocab
            n += seg
        seqs.append(t)
    off = np.zeros(n_seqs + 1, dtype=np.int64)
    off[1:] = np.cumsum([len(s) for s in seqs])
    return (np.concatenate(seqs) if seqs else np.zeros(0, np.int32)), off


def add_supersession_step(wl, more=(20, 120), own=(4, 30), seed=0):
    """A second step for a fork tree: the controller probes again while the
    earlier probes still run (the late-probe supersession of the paper's
    appendix, Algorithm 1's next retry). In every session the oldest live
    probe is freed (its blocks go back to the free queue, holding stale KV),
    the main thread decodes ``more`` further tokens (uniform) and a new probe
    forks at that point and appends ``own`` tokens (uniform). The step decodes
    one row for the main thread, the surviving probes and the new one. Drawn
    from ``numpy.random.default_rng([42, 9, seed])``; the new tokens' K and V
    from ``[42, 9, seed, seq]``."""
    rng = np.random.default_rng([42, 9, seed])
    prev = wl.steps[-1]
    si = len(wl.steps) - 1
    nid = max(t.seq for t in wl.threads) + 1
    hkv, d, dtype = wl.hkv, wl.d, wl.dtype

    def kv(key, n):
        return draw_kv([42, 9, seed, key], n, hkv, d, dtype)

    ops, seqs = [], []
    for m in [t for t in wl.threads if t.role == "main" and t.seq in prev.seqs]:
        live = [t for t in wl.threads if t.role == "probe" and t.session == m.session and t.seq in prev.seqs]
        if live:
            ops.append(("free", live[0].seq))
        add = int(rng.integers(more[0], more[1] + 1))
        length = wl.thread_len(m.seq, si)
        wl.kv_src[("s", m.seq)] = wl.kv_src[("s", m.seq)] + [([42, 9, seed, m.seq], add)]
        wl._kv_cache.pop(("s", m.seq), None)
        if wl.suffix_k is not None:
            k, v = kv(m.seq, add)
            wl.suffix_k[m.seq] = np.concatenate([wl.suffix_k[m.seq], k])
            wl.suffix_v[m.seq] = np.concatenate([wl.suffix_v[m.seq], v])
        m.suffix += add
        ops.append(("append", m.seq, add))
        n_own = int(rng.integers(own[0], own[1] + 1))
        t = Thread(seq=nid, session=m.session, role="probe", suffix=n_own, parent=m.seq, fork_len=length + add)
        wl.threads.append(t)
        wl.kv_src[("s", nid)] = [([42, 9, seed, nid], n_own)]
        if wl.suffix_k is not None:
            wl.suffix_k[nid], wl.suffix_v[nid] = kv(nid, n_own)
        ops += [("fork", m.seq, nid), ("append", nid, n_own)]
        seqs += [m.seq] + [p.seq for p in live[1:]] + [nid]
        nid += 1
    q = to_storage(rng.standard_normal((len(seqs), wl.hq, d), dtype=np.float32), dtype)
    groups = [wl.thread(s).session for s in seqs]
    wl.steps.append(Step(seqs=seqs, n_rows=[1] * len(seqs), groups=groups, q=q, ops_before=ops))
    return wl


def add_decode_steps(wl, n_steps, seed=0):
    """``n_steps`` more steps after the workload's last one, as a decode loop
    runs them: before each, every thread of the last step appends one token
    (its K and V drawn from ``[42, 10, seed, step, seq]``); each step queries
    the same threads with the same rows (the last ``n_rows`` positions of the
    grown contexts) and fresh Q from ``default_rng([42, 10, seed])``. A verify
    step's logits and drafts are kept, so its accept results stay the same.
    The pool grows by enough blocks, appended at the back of the free order
    (earlier allocations are unchanged).
    Consecutive steps can therefore reuse one plan (spork_plan_advance)."""
    rng = np.random.default_rng([42, 10, seed])
    base = wl.steps[-1]
    hkv, d, dtype = wl.hkv, wl.d, wl.dtype
    # room in the pool for the new tokens: fresh block ids at the back of the free order
    extra = len(base.seqs) * (-(-n_steps // wl.block_size) + 1)
    wl.free_order = np.concatenate([wl.free_order, np.arange(wl.num_blocks, wl.num_blocks + extra, dtype=np.int32)])
    wl.num_blocks += extra
    for i in range(n_steps):
        j = len(wl.steps)
        ops = []
        for seq in base.seqs:
            key = [42, 10, seed, j, seq]
            wl.kv_src[("s", seq)] = wl.kv_src[("s", seq)] + [(key, 1)]
            wl._kv_cache.pop(("s", seq), None)
            if wl.suffix_k is not None:
                k, v = draw_kv(key, 1, hkv, d, dtype)
                wl.suffix_k[seq] = np.concatenate([wl.suffix_k[seq], k])
                wl.suffix_v[seq] = np.concatenate([wl.suffix_v[seq], v])
            wl.thread(seq).suffix += 1
            ops.append(("append", seq, 1))
        q = to_storage(rng.standard_normal((sum(base.n_rows), wl.hq, d), dtype=np.float32), dtype)
        wl.steps.append(Step(seqs=list(base.seqs), n_rows=list(base.n_rows), groups=list(base.groups), q=q,
                             ops_before=ops, logits=base.logits, drafts=base.drafts,
                             planted_greedy=base.planted_greedy, planted_accept=base.planted_accept,
                             planted_next=base.planted_next, verify_k=base.verify_k))
    return wl
