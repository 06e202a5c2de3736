"""Host side of the C ABI, on the CPU: exports, block manager parity with the
oracle (bit-exact tables, slots, copies, refcounts and free queue), error
codes, and planner invariants."""
import copy
import ctypes
import functools
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import oracle_pool
from paper_2607_03333_amd import spork, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "spork.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spork_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(spork.LIB_PATH)
    names = _declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(spork._SIGNATURES)
    assert spork.spork_version() == 2


def _apply_both(ops, nb, bs, order):
    bm = oracle.BlockManager(nb, bs, order)
    c = spork.spork_cache_create(nb, bs, order)
    try:
        live = []
        for op in ops:
            kind = op[0]
            if kind == "new":
                assert spork.spork_seq_new(c) == bm.seq_new()
                live.append(max(bm.tables))
            elif not live:
                continue
            elif kind == "append":
                s = live[op[1] % len(live)]
                try:
                    slots, cow = bm.append(s, op[2])
                except oracle.NoBlocksError:
                    with pytest.raises(spork.SporkError) as ei:
                        spork.spork_seq_append(c, s, op[2])
                    assert ei.value.code == spork.SPORK_E_NOBLOCKS
                    continue
                gs, gc = spork.spork_seq_append(c, s, op[2])
                assert gs.tolist() == slots and gc == cow
            elif kind == "batch":
                # distinct live sequences; the oracle runs the appends one by
                # one and is restored when one of them runs out of blocks
                pairs, seen = [], set()
                for i, n in op[1]:
                    s = live[i % len(live)]
                    if s not in seen:
                        seen.add(s)
                        pairs.append((s, n))
                saved = copy.deepcopy(bm)
                try:
                    want_slots, want_cow = [], []
                    for s, n in pairs:
                        sl, cw = bm.append(s, n)
                        want_slots += sl
                        want_cow += cw
                except oracle.NoBlocksError:
                    bm = saved
                    with pytest.raises(spork.SporkError) as ei:
                        spork.spork_seq_append_batch(c, [s for s, _ in pairs], [n for _, n in pairs])
                    assert ei.value.code == spork.SPORK_E_NOBLOCKS
                else:
                    gs, gc = spork.spork_seq_append_batch(c, [s for s, _ in pairs], [n for _, n in pairs])
                    assert gs.tolist() == want_slots and gc == want_cow
            elif kind == "fork":
                p = live[op[1] % len(live)]
                assert spork.spork_fork(c, p) == bm.fork(p)
                live.append(max(bm.tables))
            elif kind == "free":
                s = live.pop(op[1] % len(live))
                bm.free_seq(s)
                spork.spork_seq_free(c, s)
            for s in live:
                assert spork.spork_block_table(c, s).tolist() == bm.table(s)
                assert spork.spork_seq_len(c, s) == bm.length(s)
            assert [spork.spork_refcount(c, b) for b in range(nb)] == bm.ref
            assert spork.spork_free_blocks(c).tolist() == bm.free_list()
    finally:
        spork.spork_cache_destroy(c)


_op = st.one_of(
    st.tuples(st.just("new")),
    st.tuples(st.just("append"), st.integers(0, 7), st.integers(0, 9)),
    st.tuples(st.just("fork"), st.integers(0, 7)),
    st.tuples(st.just("free"), st.integers(0, 7)),
    st.tuples(st.just("batch"), st.lists(st.tuples(st.integers(0, 7), st.integers(0, 9)), max_size=4)),
)


@settings(max_examples=300, deadline=None)
@given(ops=st.lists(_op, min_size=1, max_size=30), nb=st.integers(1, 12), bs=st.sampled_from([1, 2, 4, 16]),
       seed=st.integers(0, 1000))
def test_block_manager_matches_oracle(ops, nb, bs, seed):
    order = list(np.random.default_rng(seed).permutation(nb))
    _apply_both([("new",)] + ops, nb, bs, order)


def test_golden_trace_through_abi():
    import json
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "block_manager_trace.json")))
    c = spork.spork_cache_create(g["num_blocks"], g["block_size"], g["free_order"])
    for op in g["ops"]:
        if op["op"] == "new":
            assert spork.spork_seq_new(c) == op["expect_seq"]
        elif op["op"] == "fork":
            assert spork.spork_fork(c, op["parent"]) == op["expect_seq"]
        elif op["op"] == "append":
            if op.get("expect_error"):
                with pytest.raises(spork.SporkError):
                    spork.spork_seq_append(c, op["seq"], op["n"])
            else:
                slots, cow = spork.spork_seq_append(c, op["seq"], op["n"])
                assert slots.tolist() == op["expect_slots"] and [list(x) for x in cow] == op["expect_cow"]
        elif op["op"] == "free":
            spork.spork_seq_free(c, op["seq"])
    assert spork.spork_free_blocks(c).tolist() == g["final"]["free_queue"]
    assert spork.spork_block_table(c, 2).tolist() == g["final"]["tables"]["2"]
    spork.spork_cache_destroy(c)


def test_error_codes():
    with pytest.raises(spork.SporkError) as e:
        spork.spork_cache_create(4, 16, [0, 1, 1, 2])
    assert e.value.code == spork.SPORK_E_INVAL
    c = spork.spork_cache_create(4, 16)
    with pytest.raises(spork.SporkError) as e:
        spork.spork_fork(c, 3)
    assert e.value.code == spork.SPORK_E_INVAL
    s = spork.spork_seq_new(c)
    spork.spork_seq_append(c, s, 20)
    shape = spork.make_shape(4, 2, 64, 16, spork.SPORK_DTYPE_F32, 0.125)
    with pytest.raises(spork.SporkError):
        spork.spork_plan_create(c, shape, [s], [21], [0])          # more rows than tokens
    with pytest.raises(spork.SporkError):
        spork.spork_plan_create(c, spork.make_shape(4, 3, 64, 16, 0, 1.0), [s], [1], [0])
    with pytest.raises(spork.SporkError):
        spork.spork_plan_create(c, spork.make_shape(4, 2, 64, 8, 0, 1.0), [s], [1], [0])  # block size mismatch
    with pytest.raises(spork.SporkError) as e:
        spork.spork_plan_create(c, spork.make_shape(4, 2, 64, 16, 7, 1.0), [s], [1], [0])
    assert e.value.code == spork.SPORK_E_UNSUPPORTED
    p = spork.spork_plan_create(c, shape, [s], [1], [0])
    # attention with a NULL image is rejected before any launch (no GPU needed)
    with pytest.raises(spork.SporkError) as e:
        spork.spork_attn_decode(p, 0, 0, 0, 0, 0, None, None, stream=0)
    assert e.value.code in (spork.SPORK_E_INVAL, spork.SPORK_E_CAPACITY)
    # unsupported head dim for bf16
    p2 = spork.spork_plan_create(c, spork.make_shape(4, 2, 64, 16, spork.SPORK_DTYPE_BF16, 1.0), [s], [1], [0])
    with pytest.raises(spork.SporkError) as e:
        spork.spork_attn_decode(p2, 256, 256, 256, 256, 256, None, None, stream=0)
    assert e.value.code == spork.SPORK_E_UNSUPPORTED
    with pytest.raises(spork.SporkError) as e:
        spork.spork_verify_accept(None, 0, 0, 0, 0, 0, None, 0, 5, 100, 0, 1, 2, 0, 0, None, None, stream=0)
    assert e.value.code == spork.SPORK_E_UNSUPPORTED
    for h in (p, p2):
        spork.spork_plan_destroy(h)
    spork.spork_cache_destroy(c)


def test_confidence_error_codes():
    """Bad arguments of spork_probe_confidence fail on the host, before any launch."""
    conf = spork.spork_probe_confidence
    with pytest.raises(spork.SporkError) as e:
        conf(256, 7, 100, 4, 256, 1, 0.9, None, None, 256, None, None, stream=0)
    assert e.value.code == spork.SPORK_E_UNSUPPORTED
    for bad in ((256, 0, -1, 4), (256, 0, 100, -1)):          # vocab, n_rows
        with pytest.raises(spork.SporkError) as e:
            conf(bad[0], bad[1], bad[2], bad[3], 256, 1, 0.9, None, None, 256, None, None, stream=0)
        assert e.value.code == spork.SPORK_E_INVAL
    with pytest.raises(spork.SporkError) as e:                 # NULL logits
        conf(None, 0, 100, 4, 256, 1, 0.9, None, None, 256, None, None, stream=0)
    assert e.value.code == spork.SPORK_E_INVAL
    with pytest.raises(spork.SporkError) as e:                 # NULL confidence_out
        conf(256, 0, 100, 4, 256, 1, 0.9, None, None, None, None, None, stream=0)
    assert e.value.code == spork.SPORK_E_INVAL
    with pytest.raises(spork.SporkError) as e:                 # no workspace
        conf(256, 0, 100, 4, 256, 1, 0.9, None, None, 256, None, None, stream=0)
    assert e.value.code == spork.SPORK_E_CAPACITY
    # per (row, chunk) a 64-bit key and a (max, sum) float pair
    for rows, vocab in ((0, 100), (1, 151936), (40, 151936), (3, 7)):
        chunks = max(1, min(max(vocab // 8192, 1), (2048 + rows - 1) // rows if rows else 1))
        assert spork.spork_confidence_workspace_bytes(rows, vocab) == rows * chunks * 16
    # nothing to do: no launch, success
    conf(None, 0, 100, 0, None, 0, 0.9, None, None, None, None, None, stream=0)


def test_ngram_error_codes():
    """Bad arguments of spork_ngram_propose fail on the host, before any launch."""
    ng = spork.spork_ngram_propose
    for n_min, n_max, k, max_len in ((0, 3, 4, 10), (3, 2, 4, 10), (1, 33, 4, 10), (1, 3, 4097, 10),
                                     (1, 3, -1, 10), (1, 3, 4, -1), (1, 3, 4, 1 << 31)):
        with pytest.raises(spork.SporkError) as e:
            ng(256, 256, 2, max_len, n_min, n_max, k, 256, 256, None, stream=0)
        assert e.value.code == spork.SPORK_E_INVAL
    with pytest.raises(spork.SporkError) as e:                 # NULL tokens
        ng(None, 256, 2, 10, 1, 3, 4, 256, 256, None, stream=0)
    assert e.value.code == spork.SPORK_E_INVAL
    with pytest.raises(spork.SporkError) as e:                 # no workspace
        ng(256, 256, 2, 10, 1, 3, 4, 256, 256, None, stream=0)
    assert e.value.code == spork.SPORK_E_CAPACITY
    # one 64-bit key per (sequence, 2048-position chunk), at least one chunk
    for n, L, want in ((0, 10, 0), (3, 0, 24), (3, 2048, 24), (3, 2049, 48), (64, 36864, 64 * 18 * 8)):
        assert spork.spork_ngram_workspace_bytes(n, L) == want
    ng(None, None, 0, 0, 1, 3, 4, None, None, None, stream=0)   # nothing to do


def test_read_ceiling_error_codes():
    """The read-ceiling aid rejects bad arguments before any launch."""
    rc = spork.spork_read_ceiling
    for src, nbytes, grid, mode in ((None, 1 << 20, 4, 0), (256, 0, 4, 0), (256, 24, 4, 0), (264, 1 << 20, 4, 0),
                                    (256, 1 << 20, 0, 0), (256, 1 << 20, 65537, 0), (256, 1 << 20, 4, 4),
                                    (256, 1 << 20, 4, -1), (256, 3 * 16384, 2, 1), (256, 3 * 16384, 2, 3)):
        with pytest.raises(spork.SporkError) as e:
            rc(src, nbytes, grid, mode, 256, stream=0)
        assert e.value.code == spork.SPORK_E_INVAL
    with pytest.raises(spork.SporkError) as e:
        rc(256, 1 << 20, 4, 0, None, stream=0)
    assert e.value.code == spork.SPORK_E_INVAL


def test_noalloc_rejects_steps_beyond_its_scratch():
    """The no-allocation verify entry point refuses a step whose partial
    results would not fit its 64 MiB per-device scratch (the full-size probe
    prefill needs about 140 MiB) before touching the GPU, and checks its
    pointers like spork_verify_accept."""
    wl = synth.make_prefill(kv=False)
    stp = wl.steps[0]
    c = spork.spork_cache_create(wl.num_blocks, wl.block_size, wl.free_order)
    for op in stp.ops_before:
        {"new": lambda o: spork.spork_seq_new(c), "append": lambda o: spork.spork_seq_append(c, o[1], o[2]),
         "fork": lambda o: spork.spork_fork(c, o[1])}[op[0]](op)
    shape = spork.make_shape(wl.hq, wl.hkv, wl.d, wl.block_size, spork.SPORK_DTYPE_BF16, wl.sm_scale)
    p = spork.spork_plan_create(c, shape, stp.seqs, stp.n_rows, stp.groups, 256)
    try:
        assert spork.spork_plan_get_info(p)["workspace_bytes"] > (64 << 20)
        with pytest.raises(spork.SporkError) as e:
            spork.spork_verify_accept_noalloc(p, 256, 256, 256, 256, 256, 256, 256, spork.SPORK_DTYPE_BF16, 1000,
                                              256, 0, 0, 256, 256, None, stream=0)
        assert e.value.code == spork.SPORK_E_CAPACITY and "scratch" in str(e.value)
        with pytest.raises(spork.SporkError) as e:   # NULL logits with verify threads
            spork.spork_verify_accept_noalloc(None, None, None, None, None, None, None, None, spork.SPORK_DTYPE_BF16,
                                              1000, 256, 4, 2, 256, 256, None, stream=0)
        assert e.value.code == spork.SPORK_E_INVAL
    finally:
        spork.spork_plan_destroy(p)
        spork.spork_cache_destroy(c)


def _plan_for(wl, groups=None, n_cu=256):
    c = spork.spork_cache_create(wl.num_blocks, wl.block_size, wl.free_order)
    for stp in wl.steps:
        for op in stp.ops_before:
            if op[0] == "new":
                spork.spork_seq_new(c)
            elif op[0] == "append":
                spork.spork_seq_append(c, op[1], op[2])
            elif op[0] == "free":
                spork.spork_seq_free(c, op[1])
            else:
                spork.spork_fork(c, op[1])
    stp = wl.steps[-1]
    shape = spork.make_shape(wl.hq, wl.hkv, wl.d, wl.block_size,
                             spork.SPORK_DTYPE_BF16 if wl.dtype == synth.BF16 else spork.SPORK_DTYPE_F32,
                             wl.sm_scale)
    p = spork.spork_plan_create(c, shape, stp.seqs, stp.n_rows, stp.groups if groups is None else groups, n_cu)
    return c, p


def _decode_image(p):
    info = spork.spork_plan_get_info(p)
    img = spork.spork_plan_image(p)
    return info, img


@pytest.mark.parametrize("index", [0, 1, 2, 3, 4])
def test_plan_unique_bytes_match_workload(index):
    shrink = {} if index == 0 else dict(sessions=3, prefix=256, suffix=("uniform", 1, 300))
    if index == 3:
        shrink = dict(sessions=3, prefix=256, vocab=1000)
    wl = synth.make(index, **shrink)
    c, p = _plan_for(wl)
    info = spork.spork_plan_get_info(p)
    assert info["unique_kv_bytes"] == wl.unique_kv_bytes(len(wl.steps) - 1)
    assert info["n_rows"] == sum(wl.steps[-1].n_rows)
    assert info["unique_kv_bytes"] <= info["flat_kv_bytes"]
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


def _image_sections(info, img, n_out):
    """Split a plan image into its sections (256-byte aligned, in order:
    units, items, row descriptors, tables, merge offsets, partial slots,
    unit lists)."""
    raw = img.view(np.int32)
    al = lambda nbytes: -(-nbytes // 256) * 256 // 4
    nw, ni = info["n_units"], info["n_items"]
    waves = raw[: nw * 6].reshape(nw, 6)
    off = al(nw * 24)
    items = raw[off: off + ni * 8].reshape(-1, 8)
    off += al(ni * 32)
    nrow = int(items[:, 4].sum())
    rows = raw[off: off + 2 * nrow].reshape(-1, 2)
    off += al(nrow * 8)
    n_part = info["n_partials"]
    n_lists = info["attn_grid"] // 2 if info["attn_waves"] == 4 else info["attn_grid"]
    o_wg = info["image_bytes"] // 4 - al(4 * (n_lists + 1))
    o_ps = o_wg - al(4 * n_part)
    o_mo = o_ps - al(4 * (n_out + 1))
    return waves, items, rows, raw[off:o_mo], raw[o_mo: o_mo + n_out + 1], raw[o_ps: o_ps + n_part]


def _check_cover(wl, c, p, step_index=-1):
    """Decode the image: for every output (query row, head), the units that
    write one of its partials cover each visible position exactly once,
    through block-table entries equal to the thread's own table; every unit
    row writes its partial inside its output's merge range and every merge
    position is written once."""
    info, img = _decode_image(p)
    stp = wl.steps[step_index]
    hq, bs = wl.hq, wl.block_size
    n_out = sum(stp.n_rows) * hq
    waves, items, rows, tables, merge_off, part_slot = _image_sections(info, img, n_out)
    row_seq = np.repeat(np.asarray(stp.seqs), stp.n_rows)
    own = {s: spork.spork_block_table(c, s) for s in stp.seqs}
    lens = {s: spork.spork_seq_len(c, s) for s in stp.seqs}
    q_all, lo_all, top_all, slot_all = [], [], [], []
    for w in waves:
        item, lo, hi, row0, nr, part = (int(x) for x in w)
        if item < 0:
            continue
        it = items[item]
        r = rows[it[3] + row0: it[3] + row0 + nr]
        assert r.shape[0] == nr
        top = np.minimum(hi, r[:, 1] + 1)
        q_all.append(r[:, 0])
        lo_all.append(np.full(nr, lo))
        top_all.append(top)
        slot_all.append(part_slot[part: part + nr])
        seqs = row_seq[r[:, 0] // hq]
        for seq in np.unique(seqs[top > lo]):
            t = int(top[(seqs == seq) & (top > lo)].max())
            blk = np.arange(lo // bs, (t - 1) // bs + 1)
            assert np.all(blk < it[2])
            assert np.array_equal(tables[it[1] + blk], own[int(seq)][blk]), (seq, lo, t)
    q, lo, top, slot = (np.concatenate(x) for x in (q_all, lo_all, top_all, slot_all))
    # merge positions: a permutation, each inside its output's range
    assert np.array_equal(np.sort(part_slot), np.arange(info["n_partials"]))
    assert np.all((merge_off[q] <= slot) & (slot < merge_off[q + 1]))
    assert np.array_equal(np.bincount(q, minlength=n_out), np.diff(merge_off))
    # coverage: per output the non-empty ranges tile [0, pos] with no gap or overlap
    keep = top > lo
    q, lo, top = q[keep], lo[keep], top[keep]
    order = np.lexsort((lo, q))
    q, lo, top = q[order], lo[order], top[order]
    assert np.array_equal(np.unique(q), np.arange(n_out))
    first = np.r_[True, q[1:] != q[:-1]]
    last = np.r_[q[1:] != q[:-1], True]
    assert np.all(lo[first] == 0)
    assert np.all(lo[~first] == top[np.nonzero(~first)[0] - 1])
    pos = np.concatenate([np.arange(lens[s] - n, lens[s]) for s, n in zip(stp.seqs, stp.n_rows)])
    assert np.array_equal(top[last], np.repeat(pos, hq) + 1)


def _full_size(case):
    """A workload at its full size without K/V arrays (the plan needs only
    the scenario): the five benchmark workloads, the staggered fork tree and
    its supersession step, the probe prefill and the K = 50 verify."""
    if case == "tree-supersede":
        wl = oracle_pool.tight_pool(synth.add_supersession_step(synth.make_tree(kv=False)))
        assert oracle_pool.reused_blocks(wl)
        return wl
    if case == "verify-k50":
        return synth.make_named("qwen3-32b-verify", verify_k=50, kv=False)
    if case in ("tree", "prefill"):
        return synth.make_named(synth.TREE_NAME if case == "tree" else synth.PREFILL_NAME, kv=False)
    return synth.make(int(case), kv=False)


@pytest.mark.parametrize("case", ["0", "1", "2", "3", "4", "tree", "tree-supersede", "prefill", "verify-k50"])
def test_full_size_plans_cover_every_output(case):
    """Every step of every full-size workload, planned as the benchmark
    plans it (256 compute units; the 8-wave re-plan for the many-row steps):
    coverage, tables and merge ranges as in _check_cover."""
    wl = _full_size(case)
    c = spork.spork_cache_create(wl.num_blocks, wl.block_size, wl.free_order)
    shape = spork.make_shape(wl.hq, wl.hkv, wl.d, wl.block_size,
                             spork.SPORK_DTYPE_BF16 if wl.dtype == synth.BF16 else spork.SPORK_DTYPE_F32,
                             wl.sm_scale)
    try:
        for i, stp in enumerate(wl.steps):
            for op in stp.ops_before:
                if op[0] == "new":
                    spork.spork_seq_new(c)
                elif op[0] == "append":
                    spork.spork_seq_append(c, op[1], op[2])
                elif op[0] == "free":
                    spork.spork_seq_free(c, op[1])
                else:
                    spork.spork_fork(c, op[1])
            p = spork.spork_plan_create(c, shape, stp.seqs, stp.n_rows, stp.groups, 256)
            try:
                info = spork.spork_plan_get_info(p)
                if case in ("3", "prefill", "verify-k50"):   # ranges of more than 8 row tiles
                    assert info["attn_waves"] == 8
                elif wl.dtype == synth.BF16:
                    assert info["attn_waves"] == 4
                assert info["unique_kv_bytes"] == wl.unique_kv_bytes(i)
                _check_cover(wl, c, p, step_index=i)
            finally:
                spork.spork_plan_destroy(p)
    finally:
        spork.spork_cache_destroy(c)


def test_plan_covers_every_output_once_per_token():
    wl = synth.make(4, sessions=3, prefix=200, suffix=("uniform", 1, 90))
    c, p = _plan_for(wl, n_cu=4)
    _check_cover(wl, c, p)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


@pytest.mark.parametrize("prefix,stride,probes", [(256, 40, 4), (1000, 37, 3), (64, 16, 5), (300, 200, 2)])
def test_staggered_tree_plan(prefix, stride, probes):
    """Probes forked at staggered points share nested prefixes: one shared
    range per fork point, ending at the block that holds the fork point (that
    block is copied on the first write), and every output still sees each
    position once through its own blocks."""
    wl = synth.make_tree(sessions=3, prefix=prefix, stride=stride, probes=probes, probe_tokens=(1, 20),
                         main_extra=(1, 40), hq=4, hkv=2, d=64, dtype=synth.F32)
    c, p = _plan_for(wl, n_cu=8)
    info = spork.spork_plan_get_info(p)
    bs = wl.block_size
    forks = [prefix + 1 + r * stride for r in range(probes)]
    # first level: the prompt's whole blocks, then one level per later fork point
    want_shared = 3 * (forks[-1] // bs * bs)
    assert info["shared_tokens"] == want_shared
    assert info["unique_kv_bytes"] == wl.unique_kv_bytes(0)
    assert info["unique_kv_bytes"] < info["flat_kv_bytes"]
    _check_cover(wl, c, p)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


def test_tree_plan_degenerate_groups():
    """Probes forked at the same point, a probe never written after its fork,
    and a group whose members share nothing."""
    wl = synth.make_tree(sessions=2, prefix=96, stride=0, probes=3, probe_tokens=(0, 0), main_extra=(1, 9),
                         hq=4, hkv=2, d=64, dtype=synth.F32)
    c, p = _plan_for(wl, n_cu=4)
    _check_cover(wl, c, p)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)
    # every thread in one group across sessions: sessions share no block
    wl = synth.make_tree(sessions=2, prefix=64, stride=20, probes=2, probe_tokens=(1, 5), main_extra=(1, 9),
                         hq=4, hkv=2, d=64, dtype=synth.F32)
    c, p = _plan_for(wl, groups=[0] * len(wl.steps[0].seqs), n_cu=4)
    info = spork.spork_plan_get_info(p)
    assert info["unique_kv_bytes"] == wl.unique_kv_bytes(0)
    _check_cover(wl, c, p)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


@pytest.mark.parametrize("index,n_cu,shrink", [
    (4, 256, dict(sessions=6, prefix=9000, suffix=("loguniform", 1, 2000))),
    (4, 16, dict(sessions=16, prefix=20000, suffix=("loguniform", 1, 3000))),
    (3, 16, dict(sessions=3, prefix=3000, vocab=1000)),
    (2, 8, dict(sessions=4, prefix=700, suffix=("uniform", 1, 600))),
    (0, 2, {}),
])
def test_plan_lists(index, n_cu, shrink):
    """Decode the unit lists (the image's last section: list offsets into the
    unit list). bf16 plans launch 2 persistent workgroups per compute unit
    that share one list per compute unit; the lists are balanced to within
    one short piece of the per-list share (token cost plus 256 per unit),
    run longest unit first with the two row slices of a range adjacent, and
    long ranges are cut on 32-token boundaries into pieces of at most 16384
    tokens; fp32 plans run one unit per workgroup."""
    wl = synth.make(index, **shrink)
    c, p = _plan_for(wl, n_cu=n_cu)
    info, img = _decode_image(p)
    raw = img.view(np.int32)
    nu, grid = info["n_units"], info["attn_grid"]
    bf16 = wl.dtype == synth.BF16
    per_cu = 2 if info["attn_waves"] == 4 else 1
    # more than 8 row tiles in a range (the verify workload's 136 rows per KV head): 8-wave plan
    assert info["attn_waves"] == ((8 if info["max_row_tiles"] > 8 else 4) if bf16 else 1)
    assert grid == (per_cu * n_cu if bf16 else nu)
    n_lists = n_cu if bf16 else nu
    off = (info["image_bytes"] - (-(-(n_lists + 1) * 4 // 256) * 256)) // 4
    wg_off = raw[off: off + n_lists + 1]
    assert wg_off[0] == 0 and wg_off[-1] == nu and np.all(np.diff(wg_off) >= 0)
    units = raw[: nu * 6].reshape(nu, 6)
    real = units[:, 0] >= 0
    lens = units[:, 2] - units[:, 1]
    assert np.all(lens[real] > 0) and lens.max() <= 16384
    r = units[real]
    assert r[0, 5] == 0 and np.all(r[1:, 5] == r[:-1, 5] + r[:-1, 4])
    assert info["n_partials"] == int(r[-1, 5] + r[-1, 4])
    # pieces cut from one range (slice 0): contiguous, on tile boundaries,
    # and (persistent lists) at least 64 tokens but the last
    pieces = {}
    for u in r:
        if u[3] == 0:
            pieces.setdefault(int(u[0]), []).append((int(u[1]), int(u[2])))
    for item, ps in pieces.items():
        ps.sort()
        for (lo, hi), nxt in zip(ps, ps[1:]):
            assert nxt[0] == hi and hi % 32 == 0 and (hi - lo >= 64 or not bf16)
    if not bf16:
        assert np.array_equal(wg_off, np.arange(nu + 1))
        spork.spork_plan_destroy(p)
        spork.spork_cache_destroy(c)
        return
    loads = np.zeros(n_lists, dtype=np.int64)
    for x in range(n_lists):
        q = units[wg_off[x]:wg_off[x + 1]]
        ql = q[:, 2] - q[:, 1]
        assert np.all(np.diff(ql) <= 0), "list not longest first"
        loads[x] = int((ql + 256).sum())
        i = 0
        while i < len(q):  # the row slices of one piece follow each other, from row 0
            assert q[i, 3] == 0
            j = i + 1
            while j < len(q) and tuple(q[j, :3]) == tuple(q[i, :3]):
                assert q[j, 3] == q[j - 1, 3] + q[j - 1, 4]
                j += 1
            i = j
    share = -(-int(loads.sum()) // n_lists)
    longest_small = max([int(x + 256) * 2 for x in lens if int(x + 256) * 2 <= share // 2] or [0])
    assert loads.max() <= share + max(2 * (512 + 256), longest_small), (loads.max(), share)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


@pytest.mark.parametrize("shape", [dict(hq=4, hkv=2, d=64, dtype=synth.F32), dict()])
def test_probe_prefill_plan(shape):
    """Multi-row probes forked after the chain of thought: the prefix up to the
    block holding the fork point is shared by the main row and every opener
    row, each row sees each position up to its own once."""
    wl = synth.make_prefill(sessions=3, prefix=300, cot=("uniform", 1, 100), opener=(8, 50), **shape)
    c, p = _plan_for(wl, n_cu=8)
    info = spork.spork_plan_get_info(p)
    assert info["unique_kv_bytes"] == wl.unique_kv_bytes(0)
    forks = [t.fork_len for t in wl.threads if t.role == "probe"][::2]
    assert info["shared_tokens"] == sum(f // wl.block_size * wl.block_size for f in forks)
    if wl.dtype == synth.BF16:
        # openers of up to 50 rows: a shared range of up to 101 rows x 8 heads,
        # planned for 8-wave workgroups, one per compute unit
        assert info["attn_waves"] == 8 and info["attn_grid"] == 8 and info["max_row_tiles"] <= 16
    _check_cover(wl, c, p)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


def test_probe_prefill_plan_with_very_many_rows():
    """A shared range read by 70 probes of 40-50 opener rows (over 25,000
    rows per KV head, about 100 slices of 16 tiles): planned quickly, in
    slices of at most 16 tiles, and every row sees every position up to its
    own once."""
    import time
    wl = synth.make_prefill(sessions=1, prefix=600, probes=70, cot=("uniform", 1, 50), opener=(40, 50))
    t0 = time.perf_counter()
    c, p = _plan_for(wl, n_cu=8)
    assert time.perf_counter() - t0 < 5.0
    info = spork.spork_plan_get_info(p)
    assert info["attn_waves"] == 8 and info["max_row_tiles"] <= 16
    _check_cover(wl, c, p)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


def test_supersession_plan():
    """The step after a probe is freed and a new one forked: the plan's unique
    bytes and coverage hold on the reused blocks."""
    wl = synth.make_tree(sessions=3, prefix=300, stride=40, probes=3, probe_tokens=(1, 20), main_extra=(1, 30),
                         hq=4, hkv=2, d=64, dtype=synth.F32)
    synth.add_supersession_step(wl, seed=2)
    oracle_pool.tight_pool(wl)
    assert oracle_pool.reused_blocks(wl)
    c, p = _plan_for(wl, n_cu=8)
    info = spork.spork_plan_get_info(p)
    assert info["unique_kv_bytes"] == wl.unique_kv_bytes(1)
    _check_cover(wl, c, p)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


def _cache_for(wl, spare=0):
    """A cache replaying the workload's scenario, with ``spare`` more free
    blocks at the back of the free order."""
    order = np.concatenate([wl.free_order, np.arange(wl.num_blocks, wl.num_blocks + spare, dtype=np.int32)])
    c = spork.spork_cache_create(wl.num_blocks + spare, wl.block_size, order)
    for stp in wl.steps:
        for op in stp.ops_before:
            {"new": lambda o: spork.spork_seq_new(c), "append": lambda o: spork.spork_seq_append(c, o[1], o[2]),
             "fork": lambda o: spork.spork_fork(c, o[1]), "free": lambda o: spork.spork_seq_free(c, o[1])}[op[0]](op)
    return c


def test_plan_advance_refuses_what_it_cannot_absorb():
    """spork_plan_advance checks everything before it launches: no growth is a
    no-op; a freed sequence, a planned block replaced by copy-on-write, more
    new blocks than the reserve, or a grown thread without a private range
    are refused, with the plan left as it was."""
    wl = synth.make(4, sessions=2, prefix=200, suffix=("uniform", 5, 40), vocab=300, kv=False)
    stp = wl.steps[-1]
    shape = spork.make_shape(wl.hq, wl.hkv, wl.d, wl.block_size, spork.SPORK_DTYPE_BF16, wl.sm_scale)
    img_dev = 1 << 20    # a 256-aligned address; nothing is launched in this test

    def fresh(spare=0):
        c = _cache_for(wl, spare)
        return c, spork.spork_plan_create(c, shape, stp.seqs, stp.n_rows, stp.groups, 8)

    c, p = fresh()
    before = spork.spork_plan_image(p).copy()
    spork.spork_plan_advance(p, c, img_dev, stream=0)            # nothing grew: no-op
    assert np.array_equal(spork.spork_plan_image(p), before)
    spork.spork_seq_free(c, stp.seqs[1])
    with pytest.raises(spork.SporkError) as e:
        spork.spork_plan_advance(p, c, img_dev, stream=0)
    assert e.value.code == spork.SPORK_E_INVAL and "freed" in str(e.value)
    assert np.array_equal(spork.spork_plan_image(p), before)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)

    c, p = fresh(spare=200)
    main = stp.seqs[0]
    if spork.spork_seq_len(c, main) % wl.block_size == 0:
        spork.spork_seq_append(c, main, 1)                       # leave the last block partly filled
        spork.spork_plan_destroy(p)
        p = spork.spork_plan_create(c, shape, stp.seqs, stp.n_rows, stp.groups, 8)
    before = spork.spork_plan_image(p).copy()
    spork.spork_fork(c, main)                                    # shares the partial last block ...
    spork.spork_seq_append(c, main, 1)                           # ... so this append copies it
    with pytest.raises(spork.SporkError) as e:
        spork.spork_plan_advance(p, c, img_dev, stream=0)
    assert e.value.code == spork.SPORK_E_INVAL and "copy-on-write" in str(e.value)
    assert np.array_equal(spork.spork_plan_image(p), before)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)

    c, p = fresh(spare=200)
    spork.spork_seq_append(c, stp.seqs[2], 65 * wl.block_size)   # 65 new blocks: one past the reserve
    with pytest.raises(spork.SporkError) as e:
        spork.spork_plan_advance(p, c, img_dev, stream=0)
    assert e.value.code == spork.SPORK_E_CAPACITY and "reserve" in str(e.value)
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


def test_eight_wave_plan_weights_tokens_by_row_tiles():
    """8-wave plans cost a token of a row slice by the row tiles its busiest
    SIMD holds (tile t on SIMD t % 4; 1-4 tiles weigh 572, 722, 821 and 1024
    in 1/1024, from measured stage times) plus 128 tokens of start-up per
    unit: on the full-size probe prefill, whose slices hold 1-16 tiles, the
    compute units' lists are balanced under that cost (they are not under a
    plain token count), and its control words hold one 256-byte line per
    cursor (one per list plus the argmax cursor)."""
    wl = _full_size("prefill")
    c, p = _plan_for(wl)
    info, img = _decode_image(p)
    assert info["attn_waves"] == 8
    n_lists = info["attn_grid"]
    raw = img.view(np.int32)
    nu = info["n_units"]
    units = raw[: nu * 6].reshape(nu, 6)
    al = -(-(n_lists + 1) * 4 // 256) * 256 // 4
    wg_off = raw[info["image_bytes"] // 4 - al:][: n_lists + 1]
    weight = {1: 572, 2: 722, 3: 821, 4: 1024}
    cost, tokens = np.zeros(n_lists), np.zeros(n_lists)
    for x in range(n_lists):
        for u in units[wg_off[x]:wg_off[x + 1]]:
            tiles = (int(u[4]) + 15) // 16
            cost[x] += int(u[2] - u[1]) * weight[min(4, (tiles + 3) // 4)] + 128 * 1024
            tokens[x] += int(u[2] - u[1]) + 128
    assert cost.max() <= cost.mean() * 1.02, cost.max() / cost.mean()
    assert tokens.max() > tokens.mean() * 1.05  # a token count alone would not balance these lists
    assert info["control_bytes"] == (n_lists + 1) * 256
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)


def test_eight_wave_slices_by_stage_cost():
    """The K = 50 verify step's 408 rows per KV head (26 tiles) go as slices
    of 16 and 10 tiles (16 + 10: a full stage and a three-tile one per 32
    tokens), not as two near-equal 13-tile slices (four tiles on the busiest
    SIMD of each); the 136 rows of the K = 16 step stay one 9-tile slice."""
    for case, rows, want in (("verify-k50", 408, {256, 152}), ("3", 136, {136})):
        wl = _full_size(case)
        c, p = _plan_for(wl)
        info, img = _decode_image(p)
        assert info["attn_waves"] == 8
        nu = info["n_units"]
        units = img.view(np.int32)[: nu * 6].reshape(nu, 6)
        assert set(int(x) for x in units[:, 4]) == want
        # every unit's slice starts on a slice boundary of the item's rows
        assert set(int(x) for x in units[:, 3]) == ({0, 256} if case == "verify-k50" else {0})
        spork.spork_plan_destroy(p)
        spork.spork_cache_destroy(c)


def test_eight_wave_slices_each_range_at_least_stage_cost():
    """8-wave plans slice each range on its own. On the probe prefill (9-51
    row tiles per range) every item's slices are checked against brute force:
    the fewest slices (or one more) of at most 16 tiles, and no split into
    that many slices has a smaller summed stage weight (the weight of a slice
    by the tiles on its busiest SIMD: 572, 722, 821, 1024 per 1,024)."""
    weight = {1: 572, 2: 722, 3: 821, 4: 1024}
    w = lambda t: weight[(t + 3) // 4]

    @functools.lru_cache(maxsize=None)
    def best(tiles, n):  # least summed weight of n slices of 1..16 tiles adding up to tiles
        if n == 0:
            return 0 if tiles == 0 else None
        out = None
        for t in range(1, min(16, tiles - n + 1) + 1):
            rest = best(tiles - t, n - 1)
            if rest is not None and (out is None or w(t) + rest < out):
                out = w(t) + rest
        return out

    wl = _full_size("prefill")
    c, p = _plan_for(wl)
    info, img = _decode_image(p)
    assert info["attn_waves"] == 8
    units = img.view(np.int32)[: info["n_units"] * 6].reshape(-1, 6)
    slices = {}
    for it, _lo, _hi, row0, nrows, _part in units:
        slices.setdefault(int(it), set()).add((int(row0), int(nrows)))
    seen = set()
    for it, sl in slices.items():
        sl = sorted(sl)
        rows = sl[-1][0] + sl[-1][1]
        assert [r0 for r0, _ in sl] == [0] + [r0 + n for r0, n in sl[:-1]]  # contiguous, from row 0
        tiles = [(n + 15) // 16 for _, n in sl]
        total = (rows + 15) // 16
        assert sum(tiles) == total and max(tiles) <= 16
        s0 = -(-total // 16)
        assert len(tiles) in (s0, s0 + 1)
        got = sum(w(t) for t in tiles)
        assert got == min(x for x in (best(total, s0), best(total, s0 + 1)) if x is not None), (total, tiles)
        seen.add(len(tiles))
    assert seen >= {1, 2, 3}, seen   # the workload spans one to four slices per range
    spork.spork_plan_destroy(p)
    spork.spork_cache_destroy(c)
