"""Edge cases of the verify step on the GPU, against the oracle.

Through the C ABI: an accept-only call with no drafts (K = 0: the step
commits the greedy token of the one row), drafts longer than a wave (K = 100,
first mismatches past lane 63 and an all-match), the argmax over the full
151,936-entry vocabulary on maxima held by +0 and -0, natural (unplanted)
ties of coarsely rounded, saturating logits, a tie at the last two entries and an all -inf
row, and the argmax inside the persistent attention launch on a vocabulary
that is not a multiple of the 16-byte vector (the scalar scan path).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_03333_amd import runner, spork, synth
from gpu_cases import run_workload, say

pytestmark = pytest.mark.gpu
_DT = {synth.BF16: spork.SPORK_DTYPE_BF16, synth.F32: spork.SPORK_DTYPE_F32}


def accept_only(logits, dtype, drafts):
    dev = torch.device("cuda:0")
    n, k = drafts.shape
    vocab = logits.shape[1]
    lg = runner.to_device(logits, dtype, dev)
    dd = torch.from_numpy(np.ascontiguousarray(drafts, dtype=np.int32)).to(dev) if k else \
        torch.zeros(1, dtype=torch.int32, device=dev)
    acc = torch.full((n,), -1, dtype=torch.int32, device=dev)
    nxt = torch.full((n,), -1, dtype=torch.int32, device=dev)
    am = torch.full((n * (k + 1),), -1, dtype=torch.int32, device=dev)
    ws = torch.empty(spork.spork_verify_workspace_bytes(n, k, vocab) + 256, dtype=torch.uint8, device=dev)
    ws.fill_(0xFF)
    spork.spork_verify_accept(None, None, None, None, None, None, None, lg, _DT[dtype], vocab, dd, n, k, acc, nxt,
                              am, ws)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), nxt.cpu().numpy(), am.cpu().numpy()


def check(logits, dtype, drafts, tag):
    a, nx, am = accept_only(logits, dtype, drafts)
    g = oracle.argmax_rows(synth.to_f64(logits, dtype))
    wa, wn = oracle.accept_drafts(g, drafts)
    say(f"  {tag}: accept {a.tolist()[:8]} next {nx.tolist()[:4]}")
    assert np.array_equal(am, g) and np.array_equal(a, wa) and np.array_equal(nx, wn)
    return a


@pytest.mark.parametrize("dtype,vocab", [(synth.BF16, 1001), (synth.F32, 151936), (synth.BF16, 7)])
def test_no_drafts(dtype, vocab):
    rng = np.random.default_rng(vocab)
    x = rng.standard_normal((5, vocab)).astype(np.float32)
    a = check(synth.to_storage(x, dtype), dtype, np.zeros((5, 0), dtype=np.int64), f"K=0 {dtype} V={vocab}")
    assert a.tolist() == [0] * 5


def test_drafts_longer_than_a_wave():
    k, vocab, n = 100, 3000, 4
    rng = np.random.default_rng(100)
    x = rng.standard_normal((n * (k + 1), vocab)).astype(np.float32)
    greedy = rng.integers(0, vocab, size=n * (k + 1))
    x[np.arange(n * (k + 1)), greedy] = 9.0
    g = greedy.reshape(n, k + 1)
    d = rng.integers(0, vocab, size=(n, k))
    for s, m in enumerate([70, 99, 100, 63]):       # first mismatch at m (100: all match)
        d[s, :m] = g[s, :m]
        if m < k:
            d[s, m] = (g[s, m] + 1) % vocab
    a = check(synth.to_storage(x, synth.BF16), synth.BF16, d, "K=100")
    assert a.tolist() == [70, 99, 100, 63]


@pytest.mark.parametrize("dtype", [synth.BF16, synth.F32])
def test_argmax_signed_zeros_and_natural_ties_full_vocabulary(dtype):
    # -0 and +0 compare equal, so a maximum held by both goes to the lower
    # index whichever sign it has
    vocab, n, k = 151936, 3, 3
    rng = np.random.default_rng(11)
    x = -np.abs(rng.standard_normal((n * (k + 1), vocab)).astype(np.float32)) - 1.0
    x[0, 100], x[0, 5000] = -0.0, 0.0          # -0 first
    x[1, 3], x[1, 7] = 0.0, -0.0               # +0 first
    x[2, :] = -0.0
    x[2, 151000] = 0.0                         # every entry a zero: index 0
    x[3] = np.minimum(np.round(rng.standard_normal(vocab)), 3.0)   # coarse, saturating: the maximum repeats
    x[4, vocab - 2], x[4, vocab - 1] = 3.0, 3.0                # tie at the last two entries
    x[5, :] = -np.inf                          # nothing finite: index 0
    x[6] = np.minimum(np.round(rng.standard_normal(vocab) * 8.0) / 8.0, 2.0)
    x[7] = rng.standard_normal(vocab).astype(np.float32)
    st = synth.to_storage(x, dtype)
    xs = synth.to_f64(st, dtype)
    natural = [int((xs[r] == xs[r].max()).sum()) for r in (3, 6)]
    assert min(natural) > 1, natural            # the coarse rows do tie at the maximum
    assert np.signbit(xs[0, 100]) and not np.signbit(xs[0, 5000]) and np.signbit(xs[1, 7])
    g = oracle.argmax_rows(xs).reshape(n, k + 1)
    assert g[0, 0] == 100 and g[0, 1] == 3 and g[0, 2] == 0 and g[1, 0] == vocab - 2 and g[1, 1] == 0
    drafts = g[:, :k].copy()
    drafts[1, 2] = (g[1, 2] + 1) % vocab       # thread 1 stops at its third draft
    a = check(st, dtype, drafts, f"signed zeros and ties {dtype} V={vocab}")
    assert a.tolist() == [3, 2, 3]


def test_argmax_in_the_attention_tail_on_a_ragged_vocabulary():
    # vocabulary 1001: rows are not 16-byte aligned, the tail units take the
    # scalar scan path inside the persistent attention launch
    wl = synth.make(3, sessions=2, prefix=300, vocab=1001)
    run_workload(wl, "verify V=1001").close()
