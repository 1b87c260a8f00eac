"""The seeded workload generators (CPU only): determinism, length ranges, pool sizing
readings, and a block placement that hands every sequence private blocks (plus the shared
prompt's blocks in the long-document workload)."""
import numpy as np
import pytest

import workloads as W
from oracle import BlockPoolModel


@pytest.mark.parametrize("spec", W.ALL, ids=lambda s: s.name)
def test_plan_ranges_and_placement(spec):
    case = W.plan_case(spec)
    bs = spec.block_size
    seen = {}
    shared = set(case.shared_blocks.tolist())
    assert len(shared) == spec.shared_prompt_tokens // bs
    for b, bspec in zip(case.batches, spec.batches):
        assert b.n_seqs == bspec.n_seqs
        doc = b.prefix_lens - spec.shared_prompt_tokens
        if bspec.prefix.kind == "uniform":
            lo, hi = bspec.prefix.params
        else:
            lo, hi = bspec.prefix.params[2], bspec.prefix.params[3]
        assert doc.min() >= lo and doc.max() <= hi
        if bspec.kind == "decode":
            assert np.all(b.new_lens == 1)
        else:
            lo, hi = bspec.new.params
            assert b.new_lens.min() >= lo and b.new_lens.max() <= hi
        assert np.array_equal(np.diff(b.cu_new_lens), b.new_lens)
        for i in range(b.n_seqs):
            nblk = -(-int(b.prefix_lens[i] + b.new_lens[i]) // bs)
            row = b.block_tables[i]
            assert np.all(row[:nblk] >= 0) and np.all(row[nblk:] == -1)
            for blk in row[:nblk].tolist():
                if blk in shared:
                    continue
                assert blk not in seen, "a private block placed twice"
                seen[blk] = i
    needed = len(shared) + len(seen)
    kind, val = spec.pool
    if kind == "min":
        assert case.num_blocks == max(val, needed)
    elif kind == "fixed":
        assert case.num_blocks == val
    else:
        assert case.num_blocks == int(np.ceil(val * needed))


def test_same_seed_same_bytes():
    a = W.make_case(W.TINY)
    b = W.make_case(W.TINY)
    assert np.array_equal(a.pool_k, b.pool_k) and np.array_equal(a.pool_v, b.pool_v)
    assert np.array_equal(a.batches[0].q, b.batches[0].q)
    c = W.make_case(W.TINY, seed=W.TINY.seed + 100)
    assert not np.array_equal(a.pool_k, c.pool_k)


def test_stale_slots_are_nan_and_cached_slots_finite():
    case = W.make_case(W.TINY)
    bs = case.bs
    k = case.pool_k.transpose(0, 3, 1, 2, 4).reshape(case.num_blocks, bs, -1)
    v = case.pool_v.transpose(0, 3, 1, 2).reshape(case.num_blocks, bs, -1)
    for blk in range(case.num_blocks):
        n = case.valid_slots[blk]
        assert np.all(k[blk, n:] == W.BF16_NAN) and np.all(v[blk, n:] == W.BF16_NAN)
        assert not np.any(k[blk, :n] == W.BF16_NAN)


def test_lognormal_reading():
    """Long documents: median near 4096 and the clip bounds at +-2 sigma (about 4.6% clipped)."""
    rng = np.random.default_rng(0)
    from workloads.gen import _draw
    x = _draw(W.LONG_DOC_SHARED_PROMPT.batches[0].prefix, 200000, rng)
    assert abs(np.median(x) - 4096) < 60
    clipped = np.mean((x == 1024) | (x == 16384))
    assert 0.03 < clipped < 0.06


@pytest.mark.parametrize("spec", [W.TINY, W.LONG_DOC_SHARED_PROMPT.scaled(prefill=6)],
                         ids=lambda s: s.name)
def test_placement_equals_the_pool_model_allocating_in_order(spec):
    """The generator's tables are what the block pool hands out when created with the same
    free order and sequences reserve their whole length in order (the shared prompt first)."""
    case = W.plan_case(spec)
    m = BlockPoolModel(case.num_blocks, spec.block_size, free_order=case.free_order)
    parent = None
    if spec.shared_prompt_tokens:
        _, parent = m.create()
        m.reserve(parent, spec.shared_prompt_tokens)
        m.commit(parent, spec.shared_prompt_tokens)
    for b in case.batches:
        sids = []
        for i in range(b.n_seqs):
            if parent is not None:
                _, s = m.fork(parent, spec.shared_prompt_tokens)
                m.reserve(s, int(b.prefix_lens[i]) - spec.shared_prompt_tokens)
            else:
                _, s = m.create()
                m.reserve(s, int(b.prefix_lens[i]))
            m.commit(s, int(m.seqs[s].pending))
            m.reserve(s, int(b.new_lens[i]))
            sids.append(s)
        _, rows, lens = m.block_tables(sids, b.max_blocks)
        assert np.array_equal(np.asarray(rows, np.int32), b.block_tables)
        assert np.array_equal(np.asarray(lens), b.prefix_lens)
