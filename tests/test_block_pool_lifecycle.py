"""Pins of the block-pool model's lifecycle layer (prefix cache, eviction, pinning, deadlock
recovery, copy-on-write; oracle/block_pool.py) against what the paper states and what the
definitions fix, on the CPU:

  * Section 2.2's cache-miss experiment: two operators over the same table with a prefix cache
    of C tuples. Under LRU the second operator hits every tuple while the table fits and none
    once it does not (the cliff the paper measures); MRU keeps a constant number of hits
    however large the table grows, a bounded gain as Section 2.2 argues. The expected counts are worked
    out by hand in the test, not by the model.
  * Section 6: a pinned prefix is never evicted until it is unpinned; virtual pinning leaves
    eviction to the LRU order; waiting requests with none running is a deadlock whose
    recovery unpins everything and switches to virtual pinning.
  * Conservation: every block is either free or held; a block's reference count is the
    number of sequences plus cache entries holding it; refusals change nothing.
  * Copy-on-write changes exactly the shared blocks of the write range, in the writer's table
    only.
"""
import copy
import random

import pytest

from oracle import BlockPoolModel, Status
from oracle.block_pool import EXPLICIT, LRU, MRU, VIRTUAL

BS = 16


def check_invariants(m: BlockPoolModel):
    holders = [0] * m.num_blocks
    for s in m.seqs.values():
        assert len(s.blocks) == -(-(s.length + s.pending) // BS)
        assert len(set(s.blocks)) == len(s.blocks)
        for b in s.blocks:
            holders[b] += 1
    for e in m.entries.values():
        assert len(e.blocks) == -(-e.tokens // BS)
        assert len(set(e.blocks)) == len(e.blocks)
        for b in e.blocks:
            holders[b] += 1
    assert holders == m.refcount
    owned = {b for b in range(m.num_blocks) if holders[b] > 0}
    assert owned.isdisjoint(set(m.free))
    assert len(owned) + len(m.free) == m.num_blocks
    assert len(set(m.free)) == len(m.free)


def state(m):
    return copy.deepcopy((list(m.free), m.refcount,
                          {k: (s.blocks, s.length, s.pending) for k, s in m.seqs.items()},
                          {k: (e.blocks, e.tokens, e.pins, e.last_use)
                           for k, e in m.entries.items()}, m.pinning, m.eviction))


def prefill_tuple(m, key, tokens):
    """Operator 1 on one tuple: admit, compute `tokens` tokens, publish, finish."""
    _, s = m.create()
    st = m.reserve(s, tokens)
    if st != Status.OK:
        m.free_seq(s)
        return st
    m.commit(s, tokens)
    assert m.publish(s, key, tokens) == Status.OK
    m.free_seq(s)
    return Status.OK


def two_operator_hits(table, capacity_tuples, policy, blocks_per_tuple=3):
    """Section 2.2's experiment: operator 1 prefills every tuple, then operator 2 reuses each
    tuple's prefix (a hit) or recomputes it (a miss)."""
    m = BlockPoolModel(capacity_tuples * blocks_per_tuple, BS)
    m.set_eviction(policy)
    tokens = blocks_per_tuple * BS - 5  # a partly filled last block
    for t in range(table):
        assert prefill_tuple(m, t, tokens) == Status.OK
        check_invariants(m)
    hits = 0
    for t in range(table):
        st, s, n = m.attach(t)
        if st == Status.OK:
            assert n == tokens
            hits += 1
            m.free_seq(s)
        else:
            assert prefill_tuple(m, t, tokens) == Status.OK
        check_invariants(m)
    assert m.hits == hits and m.misses == table - hits
    return hits


@pytest.mark.parametrize("cap", [2, 5, 9])
def test_lru_cache_cliff_at_capacity(cap):
    # the table fits: every tuple of the second operator hits
    for table in range(1, cap + 1):
        assert two_operator_hits(table, cap, LRU) == table
    # one tuple more than fits: a sequential scan under LRU always evicts the tuple needed
    # next, so no tuple hits
    for table in (cap + 1, 2 * cap, 7 * cap + 3):
        assert two_operator_hits(table, cap, LRU) == 0


@pytest.mark.parametrize("cap", [2, 5, 9])
def test_mru_keeps_a_constant_number_of_hits(cap):
    for table in range(1, cap + 1):
        assert two_operator_hits(table, cap, MRU) == table
    # Worked by hand: after operator 1, MRU has kept tuples 0..cap-2 and the last one. In
    # operator 2 the first cap-1 tuples hit; each later miss evicts the previous recompute
    # (the most recent entry), so the last tuple survives and hits too: cap hits in all,
    # whatever the table size.
    for table in (cap + 1, 2 * cap, 7 * cap + 3):
        assert two_operator_hits(table, cap, MRU) == cap


def test_pinned_prefix_is_never_evicted_until_unpinned():
    m = BlockPoolModel(6, BS)
    assert prefill_tuple(m, "a", 32) == Status.OK  # 2 blocks each
    assert prefill_tuple(m, "b", 32) == Status.OK
    assert prefill_tuple(m, "c", 32) == Status.OK
    assert m.pin("a") == Status.OK  # the least recently used entry
    _, s = m.create()
    assert m.reserve(s, 32) == Status.OK  # evicts "b", the oldest unpinned entry
    assert set(m.entries) == {"a", "c"}
    assert m.reserve(s, 32) == Status.OK  # evicts "c"
    assert set(m.entries) == {"a"}
    before = state(m)
    assert m.reserve(s, 32) == Status.OUT_OF_BLOCKS  # only the pinned entry is left
    assert state(m) == before
    assert m.unpin("a") == Status.OK
    assert m.reserve(s, 32) == Status.OK
    assert m.entries == {}
    check_invariants(m)


def test_pin_counts_nest_and_virtual_pinning_ignores_them():
    m = BlockPoolModel(4, BS)
    assert prefill_tuple(m, 1, 32) == Status.OK
    assert prefill_tuple(m, 2, 32) == Status.OK
    assert m.pin(1) == Status.OK and m.pin(1) == Status.OK
    assert m.unpin(1) == Status.OK
    assert m.entries[1].pins == 1
    assert m.unpin(7) == Status.NOT_FOUND and m.pin(7) == Status.NOT_FOUND
    m.set_pinning(VIRTUAL)
    _, s = m.create()
    assert m.reserve(s, 32) == Status.OK  # LRU order alone: entry 1 (older) goes, pinned
    assert set(m.entries) == {2}
    assert m.unpin(2) == Status.INVALID_ARG  # never pinned
    check_invariants(m)


def test_deadlock_recovery_unpins_everything_and_switches_to_virtual():
    m = BlockPoolModel(4, BS)
    for k in (1, 2):
        assert prefill_tuple(m, k, 32) == Status.OK
        assert m.pin(k) == Status.OK
    _, s = m.create()
    assert m.reserve(s, 16) == Status.OUT_OF_BLOCKS  # every block pinned: the request waits
    # polling: requests running, or nothing waiting, is no deadlock
    assert m.check_deadlock(1, 1) == (Status.OK, 0)
    assert m.check_deadlock(0, 0) == (Status.OK, 0)
    assert m.pinning == EXPLICIT and m.entries[1].pins == 1
    assert m.check_deadlock(-1, 0)[0] == Status.INVALID_ARG
    assert m.check_deadlock(3, 0) == (Status.OK, 1)
    assert m.pinning == VIRTUAL and all(e.pins == 0 for e in m.entries.values())
    assert m.reserve(s, 16) == Status.OK  # progress: LRU eviction of entry 1
    assert set(m.entries) == {2}
    m.set_pinning(EXPLICIT)
    check_invariants(m)


def test_eviction_keeps_blocks_a_running_sequence_shares():
    m = BlockPoolModel(4, BS)
    assert prefill_tuple(m, 1, 32) == Status.OK
    assert prefill_tuple(m, 2, 32) == Status.OK
    st, user, _ = m.attach(1)  # entry 1 in use, and now the most recently used
    assert st == Status.OK
    user_blocks = list(m.seqs[user].blocks)
    _, s = m.create()
    assert m.reserve(s, 32) == Status.OK  # LRU: entry 2 goes and frees its 2 blocks
    assert set(m.entries) == {1}
    before = state(m)
    # dropping entry 1 would free nothing (user holds its blocks): refused, nothing evicted
    assert m.reserve(s, 1) == Status.OUT_OF_BLOCKS
    assert state(m) == before
    m.free_seq(user)
    assert m.reserve(s, 1) == Status.OK and m.entries == {}
    check_invariants(m)


def test_mru_eviction_may_drop_an_entry_in_use_without_taking_its_blocks():
    m = BlockPoolModel(6, BS)
    m.set_eviction(MRU)
    assert prefill_tuple(m, 1, 32) == Status.OK
    assert prefill_tuple(m, 2, 32) == Status.OK
    _, user, _ = m.attach(2)  # entry 2 becomes the most recently used
    user_blocks = list(m.seqs[user].blocks)
    _, s = m.create()
    assert m.reserve(s, 32) == Status.OK  # the 2 free blocks suffice: nothing evicted
    assert len(m.entries) == 2
    # one more block: MRU order drops entry 2 first (frees nothing: user holds it), then
    # entry 1 (frees 2)
    assert m.reserve(s, 1) == Status.OK
    assert m.entries == {} and m.evictions == 2
    assert m.seqs[user].blocks == user_blocks
    assert all(m.refcount[b] == 1 for b in user_blocks)
    check_invariants(m)


def test_eviction_is_all_or_nothing():
    m = BlockPoolModel(5, BS)
    assert prefill_tuple(m, 1, 16) == Status.OK
    assert prefill_tuple(m, 2, 16) == Status.OK
    _, s = m.create()
    before = state(m)
    assert m.reserve(s, 6 * BS) == Status.OUT_OF_BLOCKS  # 3 free + 2 evictable < 6
    assert state(m) == before
    assert m.reserve(s, 4 * BS) == Status.OK  # evicts entry 1 only
    assert set(m.entries) == {2} and m.evictions == 1
    check_invariants(m)


def test_publish_and_attach_rules():
    m = BlockPoolModel(8, BS)
    _, s = m.create()
    m.reserve(s, 40)
    assert m.publish(s, 9, 1) == Status.INVALID_ARG  # nothing committed yet
    m.commit(s, 37)
    assert m.publish(s, 9, 38) == Status.INVALID_ARG
    assert m.publish(s, 9, 0) == Status.INVALID_ARG
    assert m.publish(12345, 9, 1) == Status.NOT_FOUND
    assert m.publish(s, 9, 37) == Status.OK
    assert m.entries[9].blocks == m.seqs[s].blocks[:3]
    assert m.publish(s, 9, 16) == Status.KEY_EXISTS
    assert m.publish(s, 10, 16) == Status.OK  # a shorter prefix of the same sequence
    assert m.entries[10].blocks == m.seqs[s].blocks[:1]
    before = state(m)
    assert m.attach(11) == (Status.NOT_FOUND, 0, 0)
    assert state(m) == before and m.misses == 1
    st, c, n = m.attach(9)
    assert st == Status.OK and n == 37
    assert m.seqs[c].blocks == m.entries[9].blocks and m.seqs[c].length == 37
    assert m.seqs[c].pending == 0
    check_invariants(m)
    assert m.release(9) == Status.OK and m.release(9) == Status.NOT_FOUND
    for sid in list(m.seqs):
        m.free_seq(sid)
    assert m.release(10) == Status.OK
    assert m.num_free() == 8 and all(r == 0 for r in m.refcount)


def test_copy_on_write_of_a_partly_filled_shared_block():
    m = BlockPoolModel(10, BS)
    _, s = m.create()
    m.reserve(s, 40)
    m.commit(s, 40)
    assert m.publish(s, "p", 40) == Status.OK  # blocks 0, 1 and 2 (8 of 16 slots)
    entry_blocks = list(m.entries["p"].blocks)
    _, c, _ = m.attach("p")
    before = state(m)
    assert m.reserve(c, 4) == Status.SHARED_BLOCK_WRITE  # plain reserve refuses
    assert state(m) == before
    st, copies = m.reserve(c, 30, cow=True)  # 40 + 30 = 70 tokens: 5 blocks
    assert st == Status.OK
    assert copies == [(entry_blocks[2], 3)]  # the copy comes first off the free list
    assert m.seqs[c].blocks == entry_blocks[:2] + [3, 4, 5]
    assert m.entries["p"].blocks == entry_blocks  # the cached prefix is untouched
    assert m.seqs[s].blocks == entry_blocks  # so is the publisher's table
    assert m.refcount[entry_blocks[2]] == 2 and m.cow_copies == 1
    # a write that starts on a block boundary copies nothing
    m.commit(c, 30)
    st, copies = m.reserve(c, 10, cow=True)
    assert st == Status.OK and copies == []
    # the publisher continues its own shared last block through copy-on-write too
    st, copies = m.reserve(s, 1, cow=True)
    assert st == Status.OK and copies == [(entry_blocks[2], 6)]
    assert m.refcount[entry_blocks[2]] == 1  # only the entry holds it now
    check_invariants(m)


def test_copy_on_write_counts_its_copies_in_the_all_or_nothing_check():
    m = BlockPoolModel(4, BS)
    _, s = m.create()
    m.reserve(s, 24)
    m.commit(s, 24)
    m.publish(s, 0, 24)
    _, c, _ = m.attach(0)
    m.free_seq(s)
    # 2 blocks held by the entry and c; 2 free. Writing 24 more tokens needs one copy and
    # one growth block; writing 40 more needs one copy and two growth blocks
    before = state(m)
    assert m.reserve(c, 40, cow=True) == (Status.OUT_OF_BLOCKS, [])
    assert state(m) == before
    st, copies = m.reserve(c, 24, cow=True)
    assert st == Status.OK and len(copies) == 1 and m.num_free() == 0
    check_invariants(m)


@pytest.mark.parametrize("seed", range(6))
def test_random_lifecycle_sequences_keep_invariants(seed):
    rnd = random.Random(seed)
    n = rnd.choice([12, 40, 120])
    m = BlockPoolModel(n, BS, free_order=rnd.sample(range(n), n) if seed % 2 else None)
    if seed % 3 == 2:
        m.set_eviction(MRU)
    live, keys = [], list(range(10))
    for _ in range(600):
        op = rnd.random()
        if op < 0.1 or not live:
            live.append(m.create()[1])
        elif op < 0.35:
            s = rnd.choice(live)
            cow = rnd.random() < 0.6
            pinned = {k for k, e in m.entries.items() if e.pins and m.pinning == EXPLICIT}
            before = state(m)
            res = m.reserve(s, rnd.randint(0, 50), cow=cow)
            st = res[0] if cow else res
            if st != Status.OK:
                assert state(m) == before
            assert pinned <= set(m.entries)  # explicit pins survive every reservation
        elif op < 0.45:
            s = rnd.choice(live)
            m.commit(s, rnd.randint(0, m.seqs[s].pending))
        elif op < 0.55:
            s = rnd.choice(live)
            if m.seqs[s].length:
                m.publish(s, rnd.choice(keys), rnd.randint(1, m.seqs[s].length))
        elif op < 0.65:
            st, c, _ = m.attach(rnd.choice(keys))
            if st == Status.OK:
                live.append(c)
        elif op < 0.72:
            k = rnd.choice(keys)
            (m.pin if rnd.random() < 0.6 else m.unpin)(k)
        elif op < 0.75:
            m.release(rnd.choice(keys))
        elif op < 0.78:
            m.check_deadlock(rnd.randint(0, 2), rnd.randint(0, 1))
            if rnd.random() < 0.5:
                m.set_pinning(EXPLICIT)
        elif op < 0.85:
            s = rnd.choice(live)
            ln = m.seqs[s].length
            st, c = m.fork(s, (ln // BS) * BS)
            live.append(c)
        else:
            m.free_seq(live.pop(rnd.randrange(len(live))))
        check_invariants(m)
    for s in live:
        m.free_seq(s)
    for k in list(m.entries):
        m.release(k)
    assert m.num_free() == m.num_blocks and all(r == 0 for r in m.refcount)


def test_oracle_block_copy_moves_whole_blocks_only():
    """The copy half of copy-on-write, by brute force over a tiny pool: after copying, a
    table naming the copy reads what a table naming the source read before, and every other
    block is unchanged."""
    import numpy as np
    import oracle
    rng = np.random.default_rng(3)
    nb, hkv, d = 6, 2, 16
    pk = rng.integers(0, 1 << 16, (nb, hkv, d // 8, BS, 8), dtype=np.uint16)
    pv = rng.integers(0, 1 << 16, (nb, hkv, d, BS), dtype=np.uint16)
    ck, cv = oracle.copy_blocks(pk, pv, [(4, 1), (4, 2), (0, 5), (-1, 3), (2, 6)])
    for src, dst in [(4, 1), (4, 2), (0, 5)]:
        a = oracle.gather_seq(pk, pv, [src], BS, BS)
        b = oracle.gather_seq(ck, cv, [dst], BS, BS)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    for blk in (0, 3, 4):
        assert np.array_equal(ck[blk], pk[blk]) and np.array_equal(cv[blk], pv[blk])
    # a copy into a block that is itself a source reads the original source contents
    ck2, _ = oracle.copy_blocks(pk, pv, [(0, 1), (1, 2)])
    assert np.array_equal(ck2[2], pk[1]) and np.array_equal(ck2[1], pk[0])


def test_eviction_inside_a_copy_on_write_reservation_makes_the_block_private():
    """Regression: the shared partial block's only other holder is a cached entry that the
    reservation itself evicts to make room. The block is then private: it is written in place,
    not copied, and no block is lost."""
    m = BlockPoolModel(5, BS)
    _, s = m.create()
    m.reserve(s, 24)
    m.commit(s, 24)
    assert m.publish(s, "p", 24) == Status.OK  # 2 blocks, the second half full
    _, c, _ = m.attach("p")  # c shares both
    m.free_seq(s)
    _, s2 = m.create()
    m.reserve(s2, 16)
    m.commit(s2, 16)
    assert m.publish(s2, "q", 16) == Status.OK  # 1 block
    m.free_seq(s2)
    _, other = m.create()
    m.reserve(other, 16)  # 1 free block left
    # growing c by 20 tokens: 1 copy + 1 growth block = 2 > 1 free. LRU order: "p" (frees
    # nothing, c holds its blocks), then "q" (frees 1): enough. With "p" gone c holds its
    # partial block alone.
    st, copies = m.reserve(c, 20, cow=True)
    assert st == Status.OK and m.entries == {} and copies == []
    assert m.num_free() == 1
    check_invariants(m)
