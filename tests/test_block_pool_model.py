"""Pins of the block-pool model (oracle/block_pool.py) against invariants that the pool's
definition fixes (CPU only): conservation of blocks, reference counts equal to the number of
holders, capacity equal to the reserved length, refusals leaving state unchanged, and the
lifecycle rules the paper states (Section 2.1 block pool; Section 4 predicate pruning; Section
5.3 parents released after their children)."""
import copy
import random

import pytest

from oracle import BlockPoolModel, Status

BS = 16


def check_invariants(m: BlockPoolModel):
    holders = [0] * m.num_blocks
    for s in m.seqs.values():
        assert len(s.blocks) == -(-(s.length + s.pending) // BS)
        assert len(set(s.blocks)) == len(s.blocks)
        for b in s.blocks:
            holders[b] += 1
    assert holders == m.refcount
    owned = {b for b in range(m.num_blocks) if holders[b] > 0}
    assert owned.isdisjoint(set(m.free))
    assert len(owned) + len(m.free) == m.num_blocks
    assert len(set(m.free)) == len(m.free)


def test_ascending_and_permuted_placement():
    m = BlockPoolModel(8, BS)
    _, a = m.create()
    assert m.reserve(a, 40) == Status.OK
    assert m.seqs[a].blocks == [0, 1, 2]
    m2 = BlockPoolModel(8, BS, free_order=[5, 3, 7, 0, 1, 2, 4, 6])
    _, b = m2.create()
    assert m2.reserve(b, 17) == Status.OK
    assert m2.seqs[b].blocks == [5, 3]
    with pytest.raises(ValueError):
        BlockPoolModel(4, BS, free_order=[0, 1, 1, 2])


def test_reserve_is_all_or_nothing():
    m = BlockPoolModel(4, BS)
    _, a = m.create()
    assert m.reserve(a, 33) == Status.OK            # 3 blocks
    before = copy.deepcopy((list(m.free), m.refcount, {k: (v.blocks[:], v.length, v.pending)
                                                        for k, v in m.seqs.items()}))
    assert m.reserve(a, 32) == Status.OUT_OF_BLOCKS  # needs 2 more, 1 free
    after = (list(m.free), m.refcount, {k: (v.blocks[:], v.length, v.pending)
                                        for k, v in m.seqs.items()})
    assert before == after
    assert m.reserve(a, 31) == Status.OK             # exactly fills the pool
    assert m.num_free() == 0
    check_invariants(m)


def test_exactly_full_and_over_full_pool():
    m = BlockPoolModel(64, BS)
    sids = []
    for _ in range(8):
        _, s = m.create()
        sids.append(s)
        assert m.reserve(s, 8 * BS) == Status.OK
    assert m.num_free() == 0
    _, extra = m.create()
    assert m.reserve(extra, 1) == Status.OUT_OF_BLOCKS
    assert m.free_seq(sids[3]) == Status.OK
    assert m.num_free() == 8
    assert m.reserve(extra, 8 * BS + 1) == Status.OUT_OF_BLOCKS
    assert m.reserve(extra, 8 * BS) == Status.OK
    check_invariants(m)


def test_commit_and_partial_block_continuation():
    m = BlockPoolModel(10, BS)
    _, a = m.create()
    assert m.reserve(a, 20) == Status.OK
    assert m.commit(a, 21) == Status.INVALID_ARG
    assert m.commit(a, 20) == Status.OK
    assert m.seq_len(a) == (Status.OK, 20)
    assert m.reserve(a, 12) == Status.OK             # 32 tokens: still 2 blocks
    assert len(m.seqs[a].blocks) == 2
    assert m.reserve(a, 1) == Status.OK              # 33 tokens: a third block
    assert len(m.seqs[a].blocks) == 3
    check_invariants(m)


def test_pruned_tuple_frees_its_prefix():
    """Section 4: a predicate that drops a tuple frees the memory holding its prefix."""
    m = BlockPoolModel(12, BS)
    _, a = m.create()
    m.reserve(a, 100)
    m.commit(a, 100)
    n = m.num_free()
    assert m.free_seq(a) == Status.OK
    assert m.num_free() == n + 7
    assert m.free_seq(a) == Status.NOT_FOUND
    assert m.reserve(a, 1) == Status.NOT_FOUND


def test_parent_blocks_outlive_children_only_until_all_are_done():
    """Section 5.3: children of a Cartesian-product stage share the parent's prefix; its
    memory returns to the pool only when the parent and every child have released it."""
    m = BlockPoolModel(40, BS)
    _, parent = m.create()
    m.reserve(parent, 64)
    m.commit(parent, 64)
    kids = []
    for _ in range(17):  # the contract x hypothesis fan-out of Section 7.2's ContractNLI
        st, c = m.fork(parent, 64)
        assert st == Status.OK
        kids.append(c)
    shared = m.seqs[parent].blocks[:]
    assert all(m.refcount[b] == 18 for b in shared)
    m.free_seq(parent)
    for c in kids[:-1]:
        m.free_seq(c)
        assert all(b not in m.free for b in shared)
    m.free_seq(kids[-1])
    assert all(b in m.free for b in shared)
    check_invariants(m)


def test_write_into_shared_block_is_refused():
    m = BlockPoolModel(20, BS)
    _, parent = m.create()
    m.reserve(parent, 40)
    m.commit(parent, 40)
    assert m.fork(parent, 40)[0] == Status.INVALID_ARG  # not block aligned
    assert m.fork(parent, 48)[0] == Status.INVALID_ARG  # longer than the parent
    st, child = m.fork(parent, 32)
    assert st == Status.OK
    assert m.reserve(child, 5) == Status.OK            # starts a fresh private block
    assert m.seqs[child].blocks[:2] == m.seqs[parent].blocks[:2]
    st, c2 = m.fork(parent, 32)
    m.commit(child, 0)
    # the parent now shares its first two blocks; its own appends go to its private third block
    assert m.reserve(parent, 8) == Status.OK
    st, c3 = m.fork(c2, 32)
    assert m.free_seq(parent) == Status.OK
    # c2's last block is shared with c3 and full, so appending to c2 starts a new block: fine
    assert m.reserve(c2, 1) == Status.OK
    check_invariants(m)


def test_write_into_partially_filled_shared_block_is_refused():
    m = BlockPoolModel(20, BS)
    _, parent = m.create()
    m.reserve(parent, 32)
    m.commit(parent, 32)
    _, child = m.fork(parent, 32)
    # simulate a shorter committed length: a sequence whose last shared block is not full
    m.seqs[child].length = 30
    assert m.reserve(child, 1) == Status.SHARED_BLOCK_WRITE
    m.seqs[child].length = 32
    check_invariants(m)


@pytest.mark.parametrize("seed", range(6))
def test_random_operation_sequences_keep_invariants(seed):
    rnd = random.Random(seed)
    n = rnd.choice([16, 64, 200])
    m = BlockPoolModel(n, BS, free_order=rnd.sample(range(n), n) if seed % 2 else None)
    live = []
    for _ in range(400):
        op = rnd.random()
        if op < 0.2 or not live:
            _, s = m.create()
            live.append(s)
        elif op < 0.5:
            s = rnd.choice(live)
            before_free = m.num_free()
            st = m.reserve(s, rnd.randint(0, 70))
            if st != Status.OK:
                assert m.num_free() == before_free
        elif op < 0.65:
            s = rnd.choice(live)
            m.commit(s, rnd.randint(0, m.seqs[s].pending))
        elif op < 0.8:
            s = rnd.choice(live)
            ln = m.seqs[s].length
            st, c = m.fork(s, (ln // BS) * BS)
            assert st == Status.OK
            live.append(c)
        else:
            s = live.pop(rnd.randrange(len(live)))
            assert m.free_seq(s) == Status.OK
        check_invariants(m)
    for s in live:
        m.free_seq(s)
    assert m.num_free() == m.num_blocks
    assert all(r == 0 for r in m.refcount)


def test_block_tables_export():
    m = BlockPoolModel(10, BS, free_order=[9, 8, 7, 6, 5, 4, 3, 2, 1, 0])
    _, a = m.create()
    _, b = m.create()
    m.reserve(a, 17)
    m.commit(a, 10)
    m.reserve(b, 3)
    st, rows, lens = m.block_tables([a, b], 3)
    assert st == Status.OK
    assert rows == [[9, 8, -1], [7, -1, -1]]
    assert lens == [10, 0]
    assert m.block_tables([a], 1)[0] == Status.INVALID_ARG
    assert m.block_tables([99], 4)[0] == Status.NOT_FOUND
