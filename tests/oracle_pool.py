"""The oracle over every thread of a full-size step, in worker processes.

Each worker rebuilds the workload from its seeds without K/V arrays
(``kv=False``) and draws the K/V of the threads it is given from their own
seed streams, so nothing large crosses process boundaries. Workers run the
plain oracle (``oracle.attend`` in float64) and return each thread's output
and lse. Workers import only numpy, the oracle and the input generator; they
never touch the GPU. Started with ``spawn`` (a fresh interpreter, not a copy
of a process that uses the GPU).
"""
import multiprocessing
import os
from concurrent.futures import ProcessPoolExecutor

_WL = {}
_LIMITS = None


def build(case):
    """The workload of a full-size case, without K/V arrays. ``case`` is
    (name, keyword arguments, supersede), optionally followed by a number of
    decode steps (see decode_case)."""
    from paper_2607_03333_amd import synth
    name, kw, supersede = case[:3]
    wl = synth.make_named(name, kv=False, **kw)
    if supersede:
        wl = synth.add_supersession_step(wl)
    if len(case) > 3 and case[3]:
        synth.add_decode_steps(wl, case[3])
    return wl


def decode_case(case, n_steps):
    """The case followed by ``n_steps`` decode steps (synth.add_decode_steps)."""
    return tuple(case[:3]) + (n_steps,)


def _workload(case):
    key = repr(case)
    if key not in _WL:
        _WL.clear()
        _WL[key] = build(case)
    return _WL[key]


def _oracle_threads(case, step_index, threads):
    """(thread, first row, o, lse) for the given thread indices of a step."""
    import numpy as np

    import oracle
    from paper_2607_03333_amd import synth
    wl = _workload(case)
    st = wl.steps[step_index]
    starts = np.concatenate([[0], np.cumsum(st.n_rows)])
    res = []
    for t in threads:
        seq, n, row = st.seqs[t], st.n_rows[t], int(starts[t])
        L = wl.thread_len(seq, step_index)
        k, v = wl.context(seq, L)
        o, lse = oracle.attend(synth.to_f64(st.q[row:row + n], wl.dtype), synth.to_f64(k, wl.dtype),
                               synth.to_f64(v, wl.dtype), wl.sm_scale)
        res.append((t, row, o, lse))
    return res


def _single_threaded():
    """Worker initializer: one BLAS thread per worker (the workers already
    use every core between them)."""
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"
    import numpy  # noqa: F401  (load the BLAS, then limit the threads it already started)
    from threadpoolctl import threadpool_limits
    global _LIMITS
    _LIMITS = threadpool_limits(1)


def workers():
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


class OraclePool:
    """Submit a step's threads (grouped by session, so a worker draws each
    shared prefix once) and collect the oracle's results."""

    def __init__(self, n=None):
        ctx = multiprocessing.get_context("spawn")
        self.ex = ProcessPoolExecutor(max_workers=n or workers(), mp_context=ctx, initializer=_single_threaded)

    def submit(self, case, wl, step_index, sessions=None):
        """Futures of the oracle over the step's threads (those of ``sessions`` only, if given)."""
        st = wl.steps[step_index]
        by_session = {}
        for t, seq in enumerate(st.seqs):
            sess = wl.thread(seq).session
            if sessions is None or sess in sessions:
                by_session.setdefault(sess, []).append(t)
        return [self.ex.submit(_oracle_threads, case, step_index, ts) for ts in by_session.values()]

    def close(self):
        self.ex.shutdown(wait=True, cancel_futures=True)


def _shrunk(order, num_blocks, n):
    """The first n blocks of a free order, renumbered 0..n-1 in the same order."""
    import numpy as np
    keep = np.asarray(order[:n])
    rank = np.empty(num_blocks, dtype=np.int64)
    rank[np.sort(keep)] = np.arange(n)
    return rank[keep].astype(np.int32)


def tight_pool(wl):
    """Shrink the workload's block pool to the fewest blocks its scenario
    can run with, so that its last step must reuse blocks freed in that
    step: the pool keeps the first n blocks of the free order (the earlier
    steps take blocks in that order), renumbered 0..n-1. The oracle's
    manager replays the scenario to find n. Placement changes no result."""
    import oracle
    all_ops = [op for st in wl.steps for op in st.ops_before]
    bm = oracle.BlockManager(wl.num_blocks, wl.block_size, wl.free_order)
    _replay(bm, [op for st in wl.steps[:-1] for op in st.ops_before])
    used = wl.num_blocks - len(bm.free_list())
    assert list(bm.free_list()) == list(wl.free_order[used:]), "earlier steps freed blocks"

    def fits(n):
        try:
            _replay(oracle.BlockManager(n, wl.block_size, _shrunk(wl.free_order, wl.num_blocks, n)), all_ops)
            return True
        except oracle.NoBlocksError:
            return False

    lo, hi = used, wl.num_blocks   # fits(hi) holds: the scenario ran with the full pool
    while lo < hi:
        mid = (lo + hi) // 2
        if fits(mid):
            hi = mid
        else:
            lo = mid + 1
    wl.free_order = _shrunk(wl.free_order, wl.num_blocks, lo)
    wl.num_blocks = lo
    return wl


def reused_blocks(wl):
    """Blocks freed in the last step that some sequence holds again after it
    (oracle manager replay)."""
    import oracle
    bm = oracle.BlockManager(wl.num_blocks, wl.block_size, wl.free_order)
    _replay(bm, [op for st in wl.steps[:-1] for op in st.ops_before])
    freed = set()
    for op in wl.steps[-1].ops_before:
        before = set(bm.free_list())
        _replay(bm, [op])
        if op[0] == "free":
            freed |= set(bm.free_list()) - before
    held = {b for s in bm.tables for b in bm.table(s)}
    return sorted(freed & held)


def _replay(bm, ops):
    for op in ops:
        if op[0] == "new":
            bm.seq_new()
        elif op[0] == "append":
            bm.append(op[1], op[2])
        elif op[0] == "free":
            bm.free_seq(op[1])
        else:
            bm.fork(op[1])
