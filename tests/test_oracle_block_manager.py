"""Pins for the oracle block manager (copy-on-write fork of D1, Section 4.1).

The oracle is checked against a hand-worked trace, against invariants after
every operation of all short operation sequences, and against the closed-form
block counts of the synthetic workloads.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import BlockManager, NoBlocksError, scatter_tokens, gather_context
from oracle.kv import copy_block_prefix
from paper_2607_03333_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_trace():
    with open(os.path.join(GOLDEN, "block_manager_trace.json")) as f:
        g = json.load(f)
    bm = BlockManager(g["num_blocks"], g["block_size"], g["free_order"])
    for op in g["ops"]:
        if op["op"] == "new":
            assert bm.seq_new() == op["expect_seq"]
        elif op["op"] == "fork":
            assert bm.fork(op["parent"]) == op["expect_seq"]
        elif op["op"] == "append":
            if op.get("expect_error") == "noblocks":
                before = (dict((k, list(v)) for k, v in bm.tables.items()), dict(bm.lens), list(bm.ref), bm.free_list())
                with pytest.raises(NoBlocksError):
                    bm.append(op["seq"], op["n"])
                after = (dict((k, list(v)) for k, v in bm.tables.items()), dict(bm.lens), list(bm.ref), bm.free_list())
                assert before == after
            else:
                slots, cow = bm.append(op["seq"], op["n"])
                assert slots == op["expect_slots"]
                assert [list(c) for c in cow] == op["expect_cow"]
        elif op["op"] == "free":
            bm.free_seq(op["seq"])
    fin = g["final"]
    assert {str(k): v for k, v in bm.tables.items()} == fin["tables"]
    assert {str(k): v for k, v in bm.lens.items()} == fin["lengths"]
    assert bm.ref == fin["refcounts"]
    assert bm.free_list() == fin["free_queue"]


def _check_invariants(bm):
    refs = [0] * bm.num_blocks
    for seq, table in bm.tables.items():
        assert len(table) == -(-bm.lens[seq] // bm.block_size)
        for b in table:
            refs[b] += 1
    assert refs == bm.ref
    free = bm.free_list()
    assert len(set(free)) == len(free)
    used = {b for b in range(bm.num_blocks) if refs[b] > 0}
    assert used.isdisjoint(free)
    assert used | set(free) == set(range(bm.num_blocks))


class _ContentModel:
    """Tracks the logical token values of each sequence next to the pool.

    Tokens carry unique float values; the pool is written through the manager's
    slots (with the copy of copy-on-write applied first). After every operation
    each live sequence must read back exactly its own logical tokens.
    """

    def __init__(self, bm):
        self.bm = bm
        self.k = np.full((bm.num_blocks, 1, bm.block_size, 1), np.nan)
        self.v = np.full((bm.num_blocks, 1, 1, bm.block_size), np.nan)
        self.logical = {}
        self.counter = 0.0

    def new(self):
        s = self.bm.seq_new()
        self.logical[s] = []
        return s

    def fork(self, p):
        c = self.bm.fork(p)
        self.logical[c] = list(self.logical[p])
        return c

    def append(self, s, n):
        slots, cow = self.bm.append(s, n)
        for src, dst, nv in cow:
            copy_block_prefix(self.k, self.v, src, dst, nv)
        vals = []
        for _ in range(n):
            self.counter += 1.0
            vals.append(self.counter)
        tok = np.array(vals).reshape(n, 1, 1)
        scatter_tokens(self.k, self.v, slots, tok, -tok)
        self.logical[s].extend(vals)

    def free(self, s):
        self.bm.free_seq(s)
        del self.logical[s]

    def check(self):
        for s, vals in self.logical.items():
            k, v = gather_context(self.k, self.v, self.bm.table(s), self.bm.length(s))
            assert list(k.reshape(-1)) == vals
            assert list(v.reshape(-1)) == [-x for x in vals]


def _ops(live):
    yield ("new",)
    for s in live:
        for n in (1, 3, 6):
            yield ("append", s, n)
        yield ("fork", s)
        yield ("free", s)


def _run_all(depth, num_blocks, block_size):
    count = 0

    def rec(model, live, d):
        nonlocal count
        if d == depth:
            return
        for op in list(_ops(live)):
            bm = BlockManager(num_blocks, block_size, list(reversed(range(num_blocks))))
            m = _ContentModel(bm)
            ok_live = []
            # replay history then the new op
            for h in model:
                _apply(m, h, ok_live)
            try:
                _apply(m, op, ok_live)
            except NoBlocksError:
                _check_invariants(bm)
                m.check()
                count += 1
                continue
            _check_invariants(bm)
            m.check()
            count += 1
            rec(model + [op], list(ok_live), d + 1)

    rec([], [], 0)
    return count


def _apply(m, op, live):
    if op[0] == "new":
        live.append(m.new())
    elif op[0] == "append":
        m.append(op[1], op[2])
    elif op[0] == "fork":
        live.append(m.fork(op[1]))
    elif op[0] == "free":
        m.free(op[1])
        live.remove(op[1])


def test_all_short_sequences_keep_invariants_and_content():
    n = _run_all(depth=6, num_blocks=6, block_size=4)
    assert n > 50000


def test_exhaustion_leaves_state_unchanged():
    bm = BlockManager(3, 4)
    a = bm.seq_new()
    bm.append(a, 10)            # 3 blocks
    b = bm.fork(a)
    with pytest.raises(NoBlocksError):
        bm.append(b, 1)         # mid-block write into a shared block needs a copy target
    assert bm.table(b) == bm.table(a) and bm.length(b) == 10
    assert bm.ref == [2, 2, 2]
    bm.free_seq(a)
    slots, cow = bm.append(b, 1)  # now unshared: in place
    assert cow == [] and slots == [2 * 4 + 2]


def test_free_returns_blocks_in_table_order_fifo():
    bm = BlockManager(5, 2, [3, 0, 4, 1, 2])
    a = bm.seq_new()
    bm.append(a, 5)             # blocks 3, 0, 4
    assert bm.table(a) == [3, 0, 4]
    bm.free_seq(a)
    assert bm.free_list() == [1, 2, 3, 0, 4]


@pytest.mark.parametrize("index", [0, 1, 2, 3, 4])
def test_workload_block_counts_closed_form(index):
    """Blocks in use after the scenario equal the closed form: shared prefix
    blocks once per session plus each thread's private blocks (prefixes are
    whole blocks in every workload, so no copy-on-write happens)."""
    shrink = dict(sessions=3, prefix=64, suffix=("uniform", 1, 40)) if index in (1, 2, 3, 4) else {}
    if index == 3:
        shrink["suffix"] = ("fixed", [0])
    wl = synth.make(index, **shrink)
    bm = BlockManager(wl.num_blocks, wl.block_size, wl.free_order)
    for step in wl.steps:
        for op in step.ops_before:
            if op[0] == "new":
                assert bm.seq_new() == op[1]
            elif op[0] == "append":
                _, cow = bm.append(op[1], op[2])
                assert cow == []
            elif op[0] == "fork":
                assert bm.fork(op[1]) == op[2]
    bs = wl.block_size
    expect = sum(-(-p // bs) for p in wl.prefix_len)
    expect += sum(-(-(t.suffix + t.drafts) // bs) for t in wl.threads)
    assert wl.num_blocks - bm.num_free() == expect
    # shared prefix blocks are referenced by every member of the session
    for s, p in enumerate(wl.prefix_len):
        members = [t.seq for t in wl.threads if t.session == s]
        for b in bm.table(members[0])[: p // bs]:
            assert bm.refcount(b) == len(members)


def test_tiny_fork_counts():
    """Tiny fork: 16 shared prefix blocks (refcount 2); the main's 32 private
    tokens fill 2 blocks and its 4 verify tokens start a third (token 288 opens
    block 18); the probe's 8 tokens take 1: 20 blocks in use."""
    wl = synth.make(0)
    bm = BlockManager(wl.num_blocks, wl.block_size, wl.free_order)
    for step in wl.steps:
        for op in step.ops_before:
            if op[0] == "new":
                bm.seq_new()
            elif op[0] == "append":
                bm.append(op[1], op[2])
            else:
                bm.fork(op[1])
    assert wl.num_blocks - bm.num_free() == 16 + 3 + 1
    assert sum(1 for b in range(wl.num_blocks) if bm.refcount(b) == 2) == 16
