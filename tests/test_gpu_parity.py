"""GPU parity: the HIP path through the C ABI against the oracle, element by
element, on the five workloads (shrunk so the oracle finishes in seconds while
spanning several tiles, ragged tails and copy-on-write forks), plus the
invariants the method guarantees."""
import numpy as np
import pytest
import torch

from paper_2607_03333_amd import runner, spork, synth
import oracle_pool
from gpu_cases import compare_attention, run_workload, say

pytestmark = pytest.mark.gpu


def test_tiny_fork_full_size():
    """Tiny fork as specified: fp32, decode of main + probe, then the K=4 verify."""
    wl = synth.make(0)
    dw = run_workload(wl, "tiny-fork")
    assert dw.steps[1].accept_len.cpu().tolist() == [2]
    dw.close()


@pytest.mark.parametrize("index,shrink", [
    (1, dict(sessions=3, prefix=512, suffix=("uniform", 1, 300))),
    (2, dict(sessions=2, prefix=1024, suffix=("uniform", 1, 200))),
    (3, dict(sessions=3, prefix=700, vocab=5000)),
    (4, dict(sessions=3, prefix=1000, suffix=("loguniform", 1, 400), vocab=3000)),
])
def test_workloads_shrunk(index, shrink):
    wl = synth.make(index, **shrink)
    run_workload(wl, f"{wl.name}-shrunk").close()


def test_unaligned_fork_point_exercises_copy_on_write():
    """Prefix of 1000 tokens (not a multiple of 16): every fork's first append
    copies the shared partial block; the cascade then shares 62 whole blocks."""
    wl = synth.make(2, sessions=2, prefix=1000, suffix=("uniform", 20, 80))
    run_workload(wl, "cow").close()


def test_sharp_softmax():
    wl = synth.make(2, sessions=2, prefix=512, suffix=("uniform", 1, 100), q_gain=8.0)
    run_workload(wl, "sharp").close()


def test_single_token_contexts_and_all_rows():
    """Threads of length 1, and verify rows covering a whole short context."""
    wl = synth.make(3, sessions=2, prefix=1, vocab=600, verify_k=3)
    # prefix 1 + 3 drafts -> L = 4 with 4 rows: every row sees a different count
    run_workload(wl, "short").close()


def test_fork_without_suffix_equals_parent_bit_exact():
    wl = synth.make(2, sessions=1, prefix=777, suffix=("fixed", [0]))
    wl.steps[0].q[:] = wl.steps[0].q[0]           # same query for main and probes
    dw = run_workload(wl, "nosuffix")
    out = dw.steps[0].out.view(torch.int16)
    for t in range(1, out.shape[0]):
        assert torch.equal(out[0], out[t])
    dw.close()


def test_block_placement_does_not_change_results():
    wl = synth.make(4, sessions=2, prefix=300, suffix=("uniform", 1, 120), vocab=1000)
    dw1 = run_workload(wl, "placement-a", repeat_check=False)
    o1 = dw1.steps[0].out.view(torch.int16).clone()
    dw1.close()
    wl.free_order = np.random.default_rng(5).permutation(wl.num_blocks).astype(np.int32)
    dw2 = run_workload(wl, "placement-b", repeat_check=False)
    assert torch.equal(o1, dw2.steps[0].out.view(torch.int16))
    dw2.close()


def test_cascade_matches_flat():
    """Groups = -1 (every thread reads its whole context) against the cascade."""
    wl = synth.make(2, sessions=2, prefix=900, suffix=("uniform", 1, 64))
    dw = run_workload(wl, "cascade", repeat_check=False)
    casc = dw.steps[0].out.float()
    st = wl.steps[0]
    flat_plan = spork.spork_plan_create(dw.cache, dw.shape, st.seqs, st.n_rows, [-1] * len(st.seqs))
    info = spork.spork_plan_get_info(flat_plan)
    assert info["unique_kv_bytes"] == info["flat_kv_bytes"]
    img = torch.from_numpy(spork.spork_plan_image(flat_plan)).to(dw.device)
    out = torch.empty_like(dw.steps[0].out)
    lse = torch.empty_like(dw.steps[0].lse)
    ws = torch.empty(info["workspace_bytes"] + 256, dtype=torch.uint8, device=dw.device)
    spork.spork_workspace_clear(flat_plan, ws)  # control words zero before first use
    spork.spork_attn_decode(flat_plan, img, dw.steps[0].q, dw.k_pool, dw.v_pool, out, lse, ws)
    torch.cuda.synchronize()
    diff = (out.float() - casc).abs().max().item()
    say(f"  cascade vs flat max diff {diff:.3e}")
    assert diff <= 2e-2
    spork.spork_plan_destroy(flat_plan)
    dw.close()


def test_accept_only_mode_and_all_or_nothing_drafts():
    wl = synth.make(3, sessions=4, prefix=64, vocab=777, verify_k=5)
    st = wl.steps[0]
    g = st.planted_greedy.reshape(4, 6)
    st.drafts[0] = g[0, :5]                        # all match -> a = K, bonus token
    st.drafts[1] = (g[1, :5] + 1) % 777            # none match -> a = 0
    st.planted_accept[0], st.planted_next[0] = 5, g[0, 5]
    st.planted_accept[1], st.planted_next[1] = 0, g[1, 0]
    dw = runner.DeviceWorkload(wl)
    step = dw.prepare(0)
    step.poison()
    step.run(attention=False)
    torch.cuda.synchronize()
    assert step.accept_len.cpu().tolist()[:2] == [5, 0]
    assert np.array_equal(step.accept_len.cpu().numpy(), st.planted_accept)
    assert np.array_equal(step.next_token.cpu().numpy(), st.planted_next)
    dw.close()


@pytest.mark.parametrize("prefix,stride,probes,dtype,shape", [
    (1000, 37, 4, synth.F32, dict(hq=4, hkv=2, d=64)),      # unaligned prompt, fork points mid-block
    (4096, 200, 4, synth.BF16, dict()),                      # Qwen3-30B-A3B attention shapes
    (256, 16, 6, synth.BF16, dict(hq=64, hkv=8)),            # one fork per block, deep tree
    (640, 0, 3, synth.BF16, dict()),                         # probes forked at the same point
])
def test_staggered_fork_tree(prefix, stride, probes, dtype, shape):
    say(f"staggered tree prefix={prefix} stride={stride} probes={probes} {dtype} {shape}")
    wl = synth.make_tree(sessions=3, prefix=prefix, stride=stride, probes=probes, probe_tokens=(1, 40),
                         main_extra=(1, 60), dtype=dtype, **shape)
    dw = run_workload(wl, f"tree p{prefix} s{stride} r{probes}")
    dw.close()


@pytest.mark.parametrize("dtype,shape,opener", [
    (synth.BF16, dict(), (8, 50)),                     # Qwen3-30B-A3B shapes: 64-400 rows per KV head
    (synth.F32, dict(hq=4, hkv=2, d=64), (1, 23)),    # ragged row tiles in fp32
    (synth.BF16, dict(hq=64, hkv=8), (40, 50)),        # 320-400 rows per KV head: several row slices
])
def test_probe_prefill(dtype, shape, opener):
    """Probes prefill their forced openers (multi-row causal queries) over the
    prefix they share with the main thread, which decodes one row."""
    say(f"probe prefill {dtype} {shape} opener {opener}")
    wl = synth.make_prefill(sessions=3, prefix=700, cot=("uniform", 1, 300), opener=opener, dtype=dtype, **shape)
    dw = run_workload(wl, f"prefill {dtype} {opener}")
    dw.close()


def test_probe_prefill_very_many_rows():
    """A shared range read by 70 probes of 40-50 opener rows each: over 25,000
    rows per KV head, sliced into about 100 slices of 16 row tiles (the
    planner's fallback past its slice search)."""
    say("probe prefill, 70 probes")
    wl = synth.make_prefill(sessions=1, prefix=600, probes=70, cot=("uniform", 1, 50), opener=(40, 50))
    dw = run_workload(wl, "prefill 70 probes")
    dw.close()


def test_verify_k50():
    """Verify at the paper's draft length (K = 50): 51 causal rows per
    session, accept lengths planted up to K."""
    say("verify K=50")
    wl = synth.make(3, sessions=3, prefix=600, verify_k=50, vocab=2000)
    dw = run_workload(wl, "verify k50")
    dw.close()


@pytest.mark.parametrize("index,shrink", [
    (0, dict(block_size=32)),                                                           # fp32 decode + verify
    (4, dict(sessions=3, prefix=1000, suffix=("loguniform", 1, 400), vocab=3000, block_size=32)),
    (2, dict(sessions=2, prefix=777, suffix=("uniform", 1, 200), block_size=32)),  # fork inside a block
])
def test_block_size_32(index, shrink):
    wl = synth.make(index, **shrink)
    say(f"block size 32: {wl.name}")
    run_workload(wl, f"{wl.name}-bs32").close()


def test_staggered_tree_block_size_32():
    wl = synth.make_tree(sessions=2, prefix=640, stride=50, probes=3, probe_tokens=(1, 40), main_extra=(1, 60),
                         block_size=32)
    say("staggered tree, block size 32")
    run_workload(wl, "tree-bs32").close()


def test_probe_prefill_block_size_32():
    # more than 16 row tiles in the shared range: 8-wave workgroups, 32-token blocks
    wl = synth.make_prefill(sessions=2, prefix=700, cot=("uniform", 1, 300), opener=(40, 50), block_size=32)
    say("probe prefill, block size 32")
    run_workload(wl, "prefill-bs32").close()


@pytest.mark.parametrize("block_size", [16, 32])
def test_fp32_head_dim_128(block_size):
    # fp32 with 128-channel heads: the fp32 kernel's D = 128 instances, several
    # row slices of up to 4 tiles, and the fp32 merge at D = 128
    wl = synth.make_prefill(sessions=2, prefix=300, cot=("uniform", 1, 100), opener=(8, 30), hq=8, hkv=2, d=128,
                            dtype=synth.F32, block_size=block_size)
    say(f"fp32 head dim 128, block size {block_size}")
    run_workload(wl, f"f32-d128-bs{block_size}").close()


@pytest.mark.parametrize("dtype,shape", [(synth.F32, dict(hq=4, hkv=2, d=64)), (synth.BF16, dict())])
def test_supersession_frees_and_reforks(dtype, shape):
    """A second step after a fork tree: the oldest probe of every session is
    freed (its blocks return to the free queue with stale KV), the main thread
    decodes on and a new probe forks; the pool is as small as the scenario
    allows, so the second step's appends take the freed blocks. Both steps
    match the oracle and the block tables and free queue match the oracle
    manager."""
    wl = synth.make_tree(sessions=3, prefix=500, stride=40, probes=3, probe_tokens=(1, 30), main_extra=(1, 40),
                         dtype=dtype, **shape)
    synth.add_supersession_step(wl, seed=1)
    oracle_pool.tight_pool(wl)
    assert oracle_pool.reused_blocks(wl), "step 1 must reuse freed blocks"
    say(f"supersession {dtype}: pool {wl.num_blocks} blocks, step 1 reuses {len(oracle_pool.reused_blocks(wl))}")
    run_workload(wl, f"supersede {dtype}").close()
