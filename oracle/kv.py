"""Oracle KV placement: write tokens into the paged pools and read a context back.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Pool layout (the library's documented interface, restated here from its
definition, not imported):

* K pool ``[num_blocks, Hkv, block_size, D]``: token-major inside a block;
* V pool ``[num_blocks, Hkv, D, block_size]``: channel-major inside a block.

A token at physical slot ``s`` lives in block ``s // block_size`` at offset
``s % block_size``. A sequence's context is the concatenation, in table order,
of the valid offsets of its blocks (Section 4.1: the fork reads the parent's
prefix blocks in place).

Parity pins: a hand-built pool whose every element encodes its own
(block, head, offset, channel) index; gather after scatter returns the logical
tokens; block size and table permutation invariance.
"""

import numpy as np


def scatter_tokens(pool_k, pool_v, slots, k_tok, v_tok):
    """Write ``k_tok``/``v_tok`` (``[n, Hkv, D]``) to the given physical slots."""
    bs = pool_k.shape[2]
    for i, s in enumerate(slots):
        b, o = divmod(int(s), bs)
        pool_k[b, :, o, :] = k_tok[i]
        pool_v[b, :, :, o] = v_tok[i]


def copy_block_prefix(pool_k, pool_v, src, dst, n_valid):
    """The copy half of copy-on-write: the first ``n_valid`` offsets of ``src`` into ``dst``."""
    pool_k[dst, :, :n_valid, :] = pool_k[src, :, :n_valid, :]
    pool_v[dst, :, :, :n_valid] = pool_v[src, :, :, :n_valid]


def gather_context(pool_k, pool_v, table, length):
    """Contiguous ``K, V`` of shape ``[length, Hkv, D]`` read through ``table``."""
    bs = pool_k.shape[2]
    hkv, d = pool_k.shape[1], pool_k.shape[3]
    k = np.empty((length, hkv, d), dtype=pool_k.dtype)
    v = np.empty((length, hkv, d), dtype=pool_v.dtype)
    for i in range((length + bs - 1) // bs):
        valid = min(bs, length - i * bs)
        b = table[i]
        k[i * bs:i * bs + valid] = pool_k[b, :, :valid, :].transpose(1, 0, 2)
        v[i * bs:i * bs + valid] = pool_v[b, :, :, :valid].transpose(2, 0, 1)
    return k, v
