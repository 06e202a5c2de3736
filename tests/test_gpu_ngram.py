"""GPU parity of the n-gram (prompt-lookup) draft proposer against the oracle.

Through the C ABI: spork_ngram_propose on seeded token sequences, compared
bit-exactly (drafts, -1 padding and counts) with oracle.ngram_propose; then
the drafts feed spork_verify_accept, whose accepted lengths never pass the
real drafts.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_03333_amd import spork, synth
from gpu_cases import say

pytestmark = pytest.mark.gpu


def run_ngram(tok, off, n_min, n_max, k, max_len=None):
    dev = torch.device("cuda:0")
    n_seqs = len(off) - 1
    lens = np.diff(off)
    max_len = int(lens.max()) if max_len is None and n_seqs else (max_len or 0)
    t = torch.from_numpy(np.ascontiguousarray(tok, dtype=np.int32)).to(dev) if len(tok) else \
        torch.zeros(1, dtype=torch.int32, device=dev)
    o = torch.from_numpy(np.ascontiguousarray(off, dtype=np.int64)).to(dev)
    drafts = torch.full((max(n_seqs * k, 1),), -7, dtype=torch.int32, device=dev)
    cnt = torch.full((max(n_seqs, 1),), -7, dtype=torch.int32, device=dev)
    ws = torch.empty(max(spork.spork_ngram_workspace_bytes(n_seqs, max_len), 1), dtype=torch.uint8, device=dev)
    ws.fill_(0xA5)
    spork.spork_ngram_propose(t, o, n_seqs, max_len, n_min, n_max, k, drafts, cnt, ws)
    torch.cuda.synchronize()
    return drafts.cpu().numpy()[: n_seqs * k].reshape(n_seqs, k), cnt.cpu().numpy()[:n_seqs]


def check(tok, off, n_min, n_max, k, max_len=None, tag=""):
    d, n = run_ngram(tok, off, n_min, n_max, k, max_len)
    seqs = [tok[off[i]:off[i + 1]] for i in range(len(off) - 1)]
    wd, wn = oracle.ngram_propose(seqs, n_min, n_max, k)
    say(f"  {tag}: {len(seqs)} sequences, drafts proposed for {int((wn > 0).sum())}, mean count {wn.mean():.2f}")
    assert np.array_equal(n, wn), f"{tag}: counts differ at {np.nonzero(n != wn)[0][:8]}"
    assert np.array_equal(d, wd), f"{tag}: drafts differ at {np.nonzero((d != wd).any(axis=1))[0][:8]}"
    return d, n


@pytest.mark.parametrize("alphabet,n_min,n_max,k", [(2, 1, 3, 5), (3, 2, 4, 8), (7, 1, 1, 3), (4, 3, 5, 50),
                                                    (50, 2, 32, 16)])
def test_ngram_matches_oracle_small_alphabets(alphabet, n_min, n_max, k):
    rng = np.random.default_rng(alphabet + 10 * n_max)
    lens = [0, 1, 2, 3, 5, 17, 255, 256, 257, 2047, 2048, 2049, 2050, 4097, 6000]
    seqs = [rng.integers(0, alphabet, size=L).astype(np.int32) for L in lens]
    tok = np.concatenate(seqs)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    check(tok, off, n_min, n_max, k, tag=f"alphabet {alphabet} n {n_min}-{n_max} k {k}")


def test_ngram_repeats_and_latest_occurrence():
    # the key occurs in several chunks: the latest occurrence must win
    base = np.arange(100, 140, dtype=np.int32)
    t = np.concatenate([base, np.arange(5000, 7100, dtype=np.int32), base, np.arange(9000, 11500, dtype=np.int32),
                        base[:10], [1, 2, 3], base[:4]]).astype(np.int32)
    d, n = check(t, np.array([0, len(t)], dtype=np.int64), 2, 4, 6, tag="latest")
    assert n[0] == 6 and d[0].tolist() == base[4:10].tolist()


def test_ngram_longer_than_max_len():
    # sequences longer than max_len are scanned whole by their last chunk
    tok, off = synth.token_histories(6, [100, 5000, 9000, 2048, 3, 7000], seed=3)
    check(tok, off, 2, 4, 8, max_len=2048, tag="max_len below the lengths")
    check(tok, off, 2, 4, 8, max_len=0, tag="max_len 0")


def test_ngram_agent_histories_full_size():
    # the bench workload's histories: 64 sequences of a 32K prompt plus CoT
    say("n-gram proposer: 64 histories of 32768-36864 tokens")
    tok, off = synth.token_histories(64, (32768, 36864), seed=1)
    check(tok, off, 2, 4, 8, tag="full size")
    check(tok, off, 1, 8, 50, tag="full size, K=50")


def test_ngram_drafts_feed_verify():
    """Drafts of the proposer go straight into the accept: accepted lengths
    equal the oracle's and never pass the real draft count (the -1 padding
    never matches)."""
    dev = torch.device("cuda:0")
    tok, off = synth.token_histories(16, (300, 900), seed=5, copy_prob=0.6)
    k, vocab = 8, 1000
    tok = tok % vocab
    d, n = check(tok, off, 1, 3, k, tag="verify feed")
    rng = np.random.default_rng(9)
    logits = rng.standard_normal((16 * (k + 1), vocab)).astype(np.float32)
    # greedy tokens follow the drafts for a planted number of rows
    planted = rng.integers(0, k + 1, size=16)
    for s in range(16):
        for r in range(k + 1):
            tgt = d[s, r] if (r < planted[s] and r < k and d[s, r] >= 0) else int(rng.integers(0, vocab))
            logits[s * (k + 1) + r, tgt] = 10.0
    g = oracle.argmax_rows(logits)
    want_a, want_next = oracle.accept_drafts(g, d)
    lg = torch.from_numpy(logits).to(dev)
    dd = torch.from_numpy(d.astype(np.int32)).to(dev)
    acc = torch.full((16,), -1, dtype=torch.int32, device=dev)
    nxt = torch.full((16,), -1, dtype=torch.int32, device=dev)
    ws = torch.empty(spork.spork_verify_workspace_bytes(16, k, vocab) + 256, dtype=torch.uint8, device=dev)
    spork.spork_verify_accept(None, None, None, None, None, None, None, lg, spork.SPORK_DTYPE_F32, vocab, dd, 16, k,
                              acc, nxt, None, ws)
    torch.cuda.synchronize()
    a = acc.cpu().numpy()
    assert np.array_equal(a, want_a) and np.array_equal(nxt.cpu().numpy(), want_next)
    assert np.all(a <= n)
    say(f"  accept {a.tolist()} counts {n.tolist()}")
