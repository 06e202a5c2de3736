"""Oracle block manager: paged KV blocks shared copy-on-write between forks.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper basis: design D1 (Section 4.1) forks the probe after the main thread's
first token so that the probe's prefill is a prefix-cache hit: the probe reads
the main thread's prefix KV instead of recomputing it. The implementation
section lists prefix KV sharing between concurrent requests as a requirement of
the serving engine. A block table with reference counts and copy-on-write is
the mechanism that gives that sharing; the paper does not spell out its policy,
so the allocation rule below is this project's reading:

* free blocks form a FIFO queue seeded with a caller-given order;
* a new block is taken from the queue front when a token starts a block;
* a token written into a partially filled block that another sequence also
  references first copies that block into a fresh one (copy-on-write);
* freeing a sequence drops one reference per table entry, in table order, and a
  block whose count reaches zero goes to the back of the queue;
* an append that cannot get enough blocks raises and changes nothing.

Parity pins: brute-force enumeration of short operation sequences with
invariant checks, hand-worked traces under ``tests/golden/``, closed-form block
counts of the synthetic workloads.
"""

from collections import deque


class NoBlocksError(RuntimeError):
    """The free queue holds fewer blocks than the append needs."""


class BlockManager:
    def __init__(self, num_blocks, block_size, free_order=None):
        if num_blocks <= 0 or block_size <= 0:
            raise ValueError("num_blocks and block_size must be positive")
        order = list(range(num_blocks)) if free_order is None else [int(b) for b in free_order]
        if sorted(order) != list(range(num_blocks)):
            raise ValueError("free_order must be a permutation of 0..num_blocks-1")
        self.num_blocks = num_blocks
        self.block_size = block_size
        self.free = deque(order)
        self.ref = [0] * num_blocks
        self.tables = {}
        self.lens = {}
        self._next_seq = 0

    # -- sequences -------------------------------------------------------
    def seq_new(self):
        sid = self._next_seq
        self._next_seq += 1
        self.tables[sid] = []
        self.lens[sid] = 0
        return sid

    def _check(self, seq):
        if seq not in self.tables:
            raise KeyError(f"unknown sequence {seq}")

    def append(self, seq, n):
        """Reserve slots for ``n`` new tokens of ``seq``.

        Returns ``(slots, cow)``: the physical slot ``block * block_size +
        offset`` of each new token, and a list holding at most one
        ``(src_block, dst_block, n_valid)`` copy that must run before the new
        tokens are written.
        """
        self._check(seq)
        if n < 0:
            raise ValueError("n must be >= 0")
        bs = self.block_size
        table = self.tables[seq]
        length = self.lens[seq]
        if n == 0:
            return [], []
        # Count what the append takes from the free queue before touching state.
        shared_tail = (length % bs != 0) and self.ref[table[-1]] > 1
        fresh = sum(1 for p in range(length, length + n) if p % bs == 0)
        if shared_tail + fresh > len(self.free):
            raise NoBlocksError(f"append of {n} tokens needs {shared_tail + fresh} blocks, "
                                f"{len(self.free)} free")
        cow = []
        if shared_tail:
            src = table[-1]
            dst = self.free.popleft()
            self.ref[src] -= 1
            self.ref[dst] = 1
            table[-1] = dst
            cow.append((src, dst, length % bs))
        slots = []
        for p in range(length, length + n):
            if p % bs == 0:
                b = self.free.popleft()
                self.ref[b] = 1
                table.append(b)
            slots.append(table[p // bs] * bs + p % bs)
        self.lens[seq] = length + n
        return slots, cow

    def fork(self, parent):
        """A child sequence that shares every block of ``parent`` (no KV copied)."""
        self._check(parent)
        child = self.seq_new()
        self.tables[child] = list(self.tables[parent])
        self.lens[child] = self.lens[parent]
        for b in self.tables[child]:
            self.ref[b] += 1
        return child

    def free_seq(self, seq):
        self._check(seq)
        for b in self.tables[seq]:
            self.ref[b] -= 1
            if self.ref[b] == 0:
                self.free.append(b)
        del self.tables[seq]
        del self.lens[seq]

    # -- queries -----------------------------------------------------------
    def table(self, seq):
        self._check(seq)
        return list(self.tables[seq])

    def length(self, seq):
        self._check(seq)
        return self.lens[seq]

    def refcount(self, block):
        return self.ref[block]

    def num_free(self):
        return len(self.free)

    def free_list(self):
        return list(self.free)
