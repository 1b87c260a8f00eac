"""Plain model of the KV block pool's bookkeeping (oracle; test infrastructure only).

Semantics (each from the paper, with the readings this project takes):
  * A global pool of fixed-size blocks; blocks are taken from the pool when a request is
    admitted and returned when it completes; when too few blocks are free the request is
    deferred ("vLLM memory model", Section 2.1). Here: `reserve` is all-or-nothing and a refusal
    (OUT_OF_BLOCKS) leaves every piece of state unchanged, so the caller can defer and retry.
  * A predicate may drop a tuple, which frees the memory holding its prefix (Section 4,
    the predicate contract) -> `free`.
  * A parent task's memory is released only once all of its children are done (Section 5.3,
    Algorithm 1, Complete: children of a Cartesian-product stage are tracked as dependents of
    the parent) -> `fork` shares whole prefix blocks by reference count; a block returns to the
    free list when its last holder frees it.
  * Reading: only whole blocks are shared, so a write that would land in a block held by more
    than one sequence is refused (SHARED_BLOCK_WRITE); copy-on-write is not modelled.

Free-list order: blocks are handed out from the front of the free list, which starts as the
pool's placement order (ascending, or a caller-given permutation); a freed sequence returns its
blocks whose count drops to zero to the back of the list in table order. Sequence ids start at
1 and are never reused.
"""
from collections import deque
from enum import IntEnum


class Status(IntEnum):
    OK = 0
    INVALID_ARG = 1
    OUT_OF_BLOCKS = 2
    SHARED_BLOCK_WRITE = 3
    UNSUPPORTED_SHAPE = 4
    NOT_FOUND = 5


class _Seq:
    __slots__ = ("blocks", "length", "pending")

    def __init__(self):
        self.blocks = []
        self.length = 0   # committed tokens
        self.pending = 0  # reserved, not yet committed


class BlockPoolModel:
    def __init__(self, num_blocks, block_size, free_order=None):
        if num_blocks <= 0 or block_size <= 0:
            raise ValueError("num_blocks and block_size must be positive")
        self.num_blocks = num_blocks
        self.block_size = block_size
        order = list(range(num_blocks)) if free_order is None else [int(b) for b in free_order]
        if sorted(order) != list(range(num_blocks)):
            raise ValueError("free_order must be a permutation of 0..num_blocks-1")
        self.free = deque(order)
        self.refcount = [0] * num_blocks
        self.seqs = {}
        self.next_id = 1

    def num_free(self):
        return len(self.free)

    def create(self):
        sid = self.next_id
        self.next_id += 1
        self.seqs[sid] = _Seq()
        return Status.OK, sid

    def fork(self, parent, shared_tokens):
        if parent not in self.seqs:
            return Status.NOT_FOUND, 0
        p = self.seqs[parent]
        if shared_tokens < 0 or shared_tokens % self.block_size or shared_tokens > p.length:
            return Status.INVALID_ARG, 0
        status, sid = self.create()
        c = self.seqs[sid]
        c.blocks = p.blocks[: shared_tokens // self.block_size]
        for b in c.blocks:
            self.refcount[b] += 1
        c.length = shared_tokens
        return Status.OK, sid

    def reserve(self, sid, n):
        if sid not in self.seqs:
            return Status.NOT_FOUND
        if n < 0:
            return Status.INVALID_ARG
        if n == 0:
            return Status.OK
        s = self.seqs[sid]
        start = s.length + s.pending
        end = start + n
        first_blk = start // self.block_size
        for b in s.blocks[first_blk:]:
            if self.refcount[b] > 1:
                return Status.SHARED_BLOCK_WRITE
        need = -(-end // self.block_size) - len(s.blocks)
        if need > len(self.free):
            return Status.OUT_OF_BLOCKS
        for _ in range(need):
            b = self.free.popleft()
            self.refcount[b] = 1
            s.blocks.append(b)
        s.pending += n
        return Status.OK

    def commit(self, sid, n):
        if sid not in self.seqs:
            return Status.NOT_FOUND
        s = self.seqs[sid]
        if n < 0 or n > s.pending:
            return Status.INVALID_ARG
        s.length += n
        s.pending -= n
        return Status.OK

    def free_seq(self, sid):
        if sid not in self.seqs:
            return Status.NOT_FOUND
        s = self.seqs.pop(sid)
        for b in s.blocks:
            self.refcount[b] -= 1
            if self.refcount[b] == 0:
                self.free.append(b)
        return Status.OK

    def seq_len(self, sid):
        if sid not in self.seqs:
            return Status.NOT_FOUND, 0
        return Status.OK, self.seqs[sid].length

    def block_tables(self, sids, max_blocks):
        """Rows of physical block ids padded with -1, and committed lengths."""
        rows, lens = [], []
        for sid in sids:
            if sid not in self.seqs:
                return Status.NOT_FOUND, None, None
            s = self.seqs[sid]
            if len(s.blocks) > max_blocks:
                return Status.INVALID_ARG, None, None
            rows.append(list(s.blocks) + [-1] * (max_blocks - len(s.blocks)))
            lens.append(s.length)
        return Status.OK, rows, lens
