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
  * Reading: `fork` shares only whole blocks, and a plain `reserve` whose write range touches
    a block held by anyone else is refused (SHARED_BLOCK_WRITE). `reserve(..., cow=True)`
    instead gives the sequence a private copy of each such block (copy-on-write) and reports
    the (source, copy) pairs, whose contents the caller copies on the device.
  * Prefix cache: automatic prefix caching reuses the KV of an identical prefix and computes
    only the new suffix, and that reuse is opportunistic because a finished request's blocks
    can be reclaimed (Section 2.1). Here a sequence's first `tokens` committed tokens are
    published under a key (`publish`); the entry holds one reference on each of the
    ceil(tokens / block_size) blocks, so they outlive the sequence. `attach` turns a hit into
    a new sequence holding those blocks with length `tokens`; a miss changes nothing but the
    miss count. The last block of an entry may be partly filled; writing after it goes
    through copy-on-write.
  * Eviction: when a reservation finds too few free blocks, resident entries are dropped in
    policy order until enough blocks are free -- least recently used first by default, most
    recently used first as the alternative Section 2.2 weighs. Every entry not protected by a
    pin is a candidate; dropping it releases its references, and only blocks that no sequence
    or other entry still holds return to the free list (a running sequence keeps what it
    shares). Recency is a logical clock advanced by publish and by each hit. Reading: ties
    cannot occur (every publish and hit gets its own tick); the order is by last use alone.
    The eviction is all-or-nothing like the reservation it serves.
  * Pinning (Section 6): under explicit pinning an entry with a positive pin count is never
    evicted until it is unpinned; under virtual pinning pins protect nothing and eviction
    order alone (LRU by default) decides. Pin counts are kept in both modes.
  * Deadlock check (Section 6): requests waiting but none running is taken as a deadlock;
    recovery unpins every entry and switches to virtual pinning (the caller may switch back
    later). `release` drops an entry whatever its pins (the scheduler's own decision that the
    prefix is no longer needed).

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
    KEY_EXISTS = 7


LRU, MRU = 0, 1
EXPLICIT, VIRTUAL = 0, 1


class _Seq:
    __slots__ = ("blocks", "length", "pending")

    def __init__(self):
        self.blocks = []
        self.length = 0   # committed tokens
        self.pending = 0  # reserved, not yet committed


class _Entry:
    __slots__ = ("blocks", "tokens", "pins", "last_use")

    def __init__(self, blocks, tokens, last_use):
        self.blocks = blocks
        self.tokens = tokens
        self.pins = 0
        self.last_use = last_use


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
        self.entries = {}
        self.clock = 0
        self.eviction = LRU
        self.pinning = EXPLICIT
        self.hits = self.misses = self.evictions = self.cow_copies = 0

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

    def reserve(self, sid, n, cow=False):
        """Status, or (status, [(source, copy), ...]) when cow is set."""
        status, copies = self._reserve(sid, n, cow)
        return (status, copies) if cow else status

    def _reserve(self, sid, n, cow):
        if sid not in self.seqs:
            return Status.NOT_FOUND, []
        if n < 0:
            return Status.INVALID_ARG, []
        if n == 0:
            return Status.OK, []
        s = self.seqs[sid]
        start = s.length + s.pending
        end = start + n
        first_blk = start // self.block_size
        shared = [k for k in range(first_blk, len(s.blocks)) if self.refcount[s.blocks[k]] > 1]
        if shared and not cow:
            return Status.SHARED_BLOCK_WRITE, []
        need = -(-end // self.block_size) - len(s.blocks) + len(shared)
        if not self._make_room(need):
            return Status.OUT_OF_BLOCKS, []
        # an eviction above may have dropped a block's other holders: such a block is now
        # private and is written in place
        shared = [k for k in shared if self.refcount[s.blocks[k]] > 1]
        copies = []
        for k in shared:  # copies first, in table order
            old = s.blocks[k]
            new = self.free.popleft()
            self.refcount[new] = 1
            self.refcount[old] -= 1
            s.blocks[k] = new
            copies.append((old, new))
        self.cow_copies += len(copies)
        while len(s.blocks) * self.block_size < end:
            b = self.free.popleft()
            self.refcount[b] = 1
            s.blocks.append(b)
        s.pending += n
        return Status.OK, copies

    # -- prefix cache ---------------------------------------------------------------------
    def _candidates(self):
        """Entries that may be evicted, in eviction order."""
        keys = [k for k, e in self.entries.items() if e.pins == 0 or self.pinning == VIRTUAL]
        return sorted(keys, key=lambda k: self.entries[k].last_use,
                      reverse=(self.eviction == MRU))

    def _drop(self, key):
        e = self.entries.pop(key)
        for b in e.blocks:
            self.refcount[b] -= 1
            if self.refcount[b] == 0:
                self.free.append(b)

    def _make_room(self, need):
        if need <= len(self.free):
            return True
        # what would evicting the first k candidates free? (all-or-nothing)
        order = self._candidates()
        left = list(self.refcount)
        freed, k = 0, 0
        while len(self.free) + freed < need and k < len(order):
            for b in self.entries[order[k]].blocks:
                left[b] -= 1
                if left[b] == 0:
                    freed += 1
            k += 1
        if len(self.free) + freed < need:
            return False
        for key in order[:k]:
            self._drop(key)
        self.evictions += k
        return True

    def _tick(self):
        self.clock += 1
        return self.clock

    def publish(self, sid, key, tokens):
        if sid not in self.seqs:
            return Status.NOT_FOUND
        s = self.seqs[sid]
        if tokens <= 0 or tokens > s.length:
            return Status.INVALID_ARG
        if key in self.entries:
            return Status.KEY_EXISTS
        blocks = s.blocks[: -(-tokens // self.block_size)]
        for b in blocks:
            self.refcount[b] += 1
        self.entries[key] = _Entry(list(blocks), tokens, self._tick())
        return Status.OK

    def lookup(self, key):
        """Tokens cached under key, or 0 when absent; changes nothing (no hit, no recency)."""
        e = self.entries.get(key)
        return 0 if e is None else e.tokens

    def attach(self, key):
        """(status, sequence id, tokens): a hit makes a new sequence holding the entry."""
        if key not in self.entries:
            self.misses += 1
            return Status.NOT_FOUND, 0, 0
        e = self.entries[key]
        _, sid = self.create()
        s = self.seqs[sid]
        s.blocks = list(e.blocks)
        s.length = e.tokens
        for b in e.blocks:
            self.refcount[b] += 1
        e.last_use = self._tick()
        self.hits += 1
        return Status.OK, sid, e.tokens

    def pin(self, key):
        if key not in self.entries:
            return Status.NOT_FOUND
        self.entries[key].pins += 1
        return Status.OK

    def unpin(self, key):
        if key not in self.entries:
            return Status.NOT_FOUND
        if self.entries[key].pins == 0:
            return Status.INVALID_ARG
        self.entries[key].pins -= 1
        return Status.OK

    def release(self, key):
        if key not in self.entries:
            return Status.NOT_FOUND
        self._drop(key)
        return Status.OK

    def set_eviction(self, policy):
        if policy not in (LRU, MRU):
            return Status.INVALID_ARG
        self.eviction = policy
        return Status.OK

    def set_pinning(self, mode):
        if mode not in (EXPLICIT, VIRTUAL):
            return Status.INVALID_ARG
        self.pinning = mode
        return Status.OK

    def check_deadlock(self, waiting, running):
        """(status, recovered): waiting > 0 and running == 0 unpins all, switches to virtual."""
        if waiting < 0 or running < 0:
            return Status.INVALID_ARG, 0
        if waiting > 0 and running == 0:
            for e in self.entries.values():
                e.pins = 0
            self.pinning = VIRTUAL
            return Status.OK, 1
        return Status.OK, 0

    def stats(self):
        held_by_seq = {b for s in self.seqs.values() for b in s.blocks}
        cached = {b for e in self.entries.values() for b in e.blocks} - held_by_seq
        return {"num_free": len(self.free), "num_entries": len(self.entries),
                "cached_blocks": len(cached),
                "pinned_entries": sum(1 for e in self.entries.values() if e.pins > 0),
                "hits": self.hits, "misses": self.misses, "evictions": self.evictions,
                "cow_copies": self.cow_copies, "eviction": self.eviction,
                "pinning": self.pinning}

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
