"""CPU oracle for SPORK's forked-decode hot path.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything under ``oracle/``. The
product path (``paper_2607_03333_amd``) never imports it and shares no code with it.

Plain, slow, obviously correct: Python integers for the block manager, NumPy in
float64 for attention, argmax and accept. Every function cites the part of the
paper it follows (SPORK, arXiv 2607.03333):

* block manager: the copy-on-write block table behind the prefix-cache fork of
  design D1 (Section 4.1) -- the probe reuses the main thread's prefix KV.
* attention: softmax attention of the main and probe rows over their paged
  context, with a bottom-right causal rule for multi-row (verify) threads
  (Section 4.3, step 2; greedy decoding, Section 6.1 "Setup").
* argmax + accept: greedy target tokens and the longest draft prefix that
  matches them (Section 4.3, steps 2-3; Appendix B).
* confidence: the top-1 log-probability of each probe position and the D2
  gate over the tool-name span (Section 4.2).
* ngram: the prompt-lookup draft proposer of the engine's n-gram speculative
  decoding, the drafts' second source beside the probe body (Sections 4.3,
  6.1).

Parity status of each function is stated in its module header.
"""

from .block_manager import BlockManager, NoBlocksError
from .kv import scatter_tokens, gather_context
from .attention import attend, attend_batch
from .accept import argmax_rows, accept_drafts
from .confidence import top1_logprob, span_confidence, confidence_gate
from .ngram import ngram_propose, ngram_propose_one

__all__ = [
    "BlockManager", "NoBlocksError", "scatter_tokens", "gather_context",
    "attend", "attend_batch", "argmax_rows", "accept_drafts",
    "top1_logprob", "span_confidence", "confidence_gate",
    "ngram_propose", "ngram_propose_one",
]
